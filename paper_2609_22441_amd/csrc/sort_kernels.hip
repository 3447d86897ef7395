// Alg. 1 Step 1 on the device (Connected Content Retriever §3.1): sort each viewer's affinity
// records by author id and move their feature rows with them.
//
// A record is sorted as an element that orders by (key, input position). That order is unique,
// so any correct sort is stable. Elements take one of two forms, chosen on the device for the
// whole call:
//   * packed, 8 bytes: ((key - kmin) << pbits) | (position within the viewer), when the span of
//     the call's keys leaves room for pbits position bits (pbits covers the largest viewer);
//   * wide, 16 bytes: (key, flat input position), for any keys.
// Every call starts with the key range (per-workgroup slots, reduced by a plan kernel). Then one
// of two methods, chosen on the host (by call size, or by the caller):
//
// Merge (calls below kSortRadixMinRecords records): tiles of kTile records per viewer; a block
// sort per tile (every thread sorts kEpt records in registers with a bitonic network, then
// merge-path rounds in LDS double the sorted runs), then merge rounds within each viewer. A
// viewer's last pass writes the sorted keys and copies the rows.
//
// Radix (larger calls): the keys are ordered on kbits = the bit length of kmax - kmin, in
// P = ceil(kbits / 9) digits of D = ceil(kbits / P) <= 9 bits, least significant first (a
// stable LSD radix sort: no comparison of whole keys, equal keys keep their input order).
//   1. small viewers (at most kTile records): one workgroup sorts the viewer in LDS as above and
//      writes its sorted keys and, for each output position, the input position of its record;
//      for a multi-tile viewer the same kernel clears its digit histogram.
//   2. histogram: for every tile of a multi-tile viewer (tiles of 8192 packed or 4096 wide
//      records, listed by the plan), the counts of each digit value of every pass, added into
//      the viewer's histogram; each tile's descriptor for the passes.
//   3. one kernel per digit (the launches past P return at once): every tile ranks its records
//      by the digit (stable, in LDS), learns how many records of each digit value the viewer's
//      earlier tiles hold from the tiles' published counts (decoupled look-back), and scatters
//      its records to viewer start + records of smaller digit values + that count + rank. The
//      last digit's pass writes the sorted keys and the input positions.
//   4. gather: every output row copied from its record's input row.
// Tiles take their index from a counter in claim order, so every earlier tile of a viewer is
// held by a running workgroup and publishes its counts without waiting for later ones.
#include <stdint.h>

#include <mutex>

#include <hip/hip_runtime.h>

#include "join_internal.h"

namespace ccj {
namespace {

constexpr int kTile = 4096;                       // records per tile
constexpr int kThreads = 512;                     // threads per workgroup
constexpr int kWaves = kThreads / 64;
constexpr int kEpt = kTile / kThreads;            // records per thread (8)
constexpr int kLdsElems = kTile + kTile / kEpt;   // padded LDS tile of the small-viewer sort
constexpr int kDigitBits = 9;                     // widest digit
constexpr int kRadix = 1 << kDigitBits;           // values of one digit (512 = kThreads)
constexpr int kMaxPasses = 8;                     // 64-bit key spans
constexpr int kDirectPasses = 3;                  // key spans up to 27 bits
constexpr unsigned kLoopGrid = 256;               // workgroups of the later passes

typedef unsigned int chunk_t __attribute__((ext_vector_type(4)));

// Shared by every kernel of one call: the key range (written by the plan) and the number of
// position bits a packed element needs.
struct Codec {
    const int64_t *range;   // {min key, max key} in the workspace
    int32_t pbits;
    int32_t max_passes;     // digit passes launched (from the caller's bound on the key span)
};

struct Wide {
    struct T {
        int64_t key;
        int64_t f;    // flat input position
    };
    int64_t kmin;
    static constexpr int kRadixEpt = 8;     // records per thread of a digit pass (64 KiB tile)
    __device__ static bool less(const T &a, const T &b) {
        return a.key != b.key ? a.key < b.key : a.f < b.f;
    }
    __device__ static T pad() { return T{INT64_MAX, INT64_MAX}; }
    // c ? x : y field by field (a select of the whole struct is lowered through scratch memory).
    __device__ static T sel(bool c, const T &x, const T &y) {
        return T{c ? x.key : y.key, c ? x.f : y.f};
    }
    __device__ T make(int64_t key, int64_t f, int64_t) const { return T{key, f}; }
    __device__ int64_t key(const T &e) const { return e.key; }
    __device__ int64_t src(const T &e, int64_t) const { return e.f; }
    __device__ uint32_t digit(const T &e, int shift, uint32_t mask) const {
        return (uint32_t)(((uint64_t)e.key - (uint64_t)kmin) >> shift) & mask;
    }
};

struct Packed {
    typedef uint64_t T;
    int64_t kmin;
    int32_t pbits;
    static constexpr int kRadixEpt = 16;    // records per thread of a digit pass (64 KiB tile)
    __device__ static bool less(T a, T b) { return a < b; }
    __device__ static T pad() { return ~(uint64_t)0; }    // above every packed record
    __device__ static T sel(bool c, T x, T y) { return c ? x : y; }
    __device__ T make(int64_t key, int64_t f, int64_t kb) const {
        return (((uint64_t)key - (uint64_t)kmin) << pbits) | (uint64_t)(f - kb);
    }
    __device__ int64_t key(T e) const { return (int64_t)((e >> pbits) + (uint64_t)kmin); }
    __device__ int64_t src(T e, int64_t kb) const {
        return kb + (int64_t)(e & ((((uint64_t)1) << pbits) - 1));
    }
    // pbits + shift < 64: the packed form holds kbits <= 64 - pbits key bits, and every digit
    // starts below kbits.
    __device__ uint32_t digit(T e, int shift, uint32_t mask) const {
        return (uint32_t)(e >> (pbits + shift)) & mask;
    }
};

// Packed elements are usable when key - kmin < 2^(64 - pbits) - 1 for every key (the largest
// value stays free for padding). Every kernel evaluates this on the same range.
__device__ __forceinline__ bool packs(int64_t kmin, int64_t kmax, int32_t pbits) {
    if (kmax < kmin)
        return true;                                    // no keys
    const uint64_t span = (uint64_t)kmax - (uint64_t)kmin;
    return span < (((uint64_t)1) << (64 - pbits)) - 1;
}

__device__ __forceinline__ bool use_packed(const Codec &c, int64_t &kmin) {
    kmin = c.range[0];
    return packs(kmin, c.range[1], c.pbits);
}

// The call's digits: P passes of D <= kDigitBits bits over the bit length of kmax - kmin (one
// pass of one always-zero bit when every key is equal). P * D >= kbits and (P - 1) * D < kbits;
// P <= kMaxPasses for 64-bit spans. When the keys span more bits than the launched passes
// cover (a caller's bound that does not hold), those passes take full-width digits: the low
// max_passes * kDigitBits bits of key - kmin are ordered, the rest are not.
struct Digits {
    int P, D;
    uint32_t mask;
};

__device__ __forceinline__ Digits digits_of(const Codec &c) {
    const int64_t kmin = c.range[0], kmax = c.range[1];
    const uint64_t span = kmax < kmin ? 0 : (uint64_t)kmax - (uint64_t)kmin;
    const int kbits = span ? 64 - __clzll(span) : 0;
    const int P = kbits ? (kbits + kDigitBits - 1) / kDigitBits : 1;
    if (P > c.max_passes)
        return Digits{c.max_passes, kDigitBits, (1u << kDigitBits) - 1};
    const int D = kbits ? (kbits + P - 1) / P : 1;
    return Digits{P, D, (1u << D) - 1};
}

__device__ __forceinline__ int pidx(int i) { return i + i / kEpt; }

__device__ __forceinline__ void lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ int64_t clampk(int64_t v, int64_t hi) {
    return v < 0 ? 0 : (v > hi ? hi : v);
}

// Segment [kb, ke) of viewer v, offsets clamped to [0, total] and made non-decreasing.
__device__ __forceinline__ void segment(const int64_t *off, int64_t total, int64_t v, int64_t &kb,
                                        int64_t &ke) {
    kb = clampk(off[v], total);
    ke = max(kb, clampk(off[v + 1], total));
}

__device__ __forceinline__ int64_t tiles_of(int64_t n) { return (n + kTile - 1) / kTile; }

__device__ __forceinline__ int rounds_of(int64_t tiles) {
    int r = 0;
    while (((int64_t)1 << r) < tiles)
        ++r;
    return r;
}

// Records per tile of the digit passes: 8192 packed or 4096 wide elements (64 KiB of LDS).
__device__ __forceinline__ int radix_tile(bool packed) {
    return (packed ? Packed::kRadixEpt : Wide::kRadixEpt) * kThreads;
}

// Tiles of a viewer with n records in the list of multi-tile viewers' tiles (tiles of
// radix_tile records): none for a viewer that the small-viewer sort takes whole.
__device__ __forceinline__ int64_t multi_tiles(int64_t n, int tile) {
    return n > kTile ? (n + tile - 1) / tile : 0;
}

// Largest v in [0, B) with tile_off[v] <= t (tile_off non-decreasing, tile_off[0] = 0), found by
// the whole workgroup (call it uniformly). Each round every thread probes one of kThreads
// evenly spaced viewers; the probes at or below t are a prefix, and its length narrows the range
// kThreads-fold. Up to kThreads viewers take one round of independent loads instead of a chain
// of ~log2(B) dependent ones.
__device__ __forceinline__ int64_t owner(const int64_t *tile_off, int64_t B, int64_t t) {
    int64_t lo = 0, hi = B - 1;                   // tile_off[lo] <= t; the answer is in [lo, hi]
    while (lo < hi) {
        const int64_t step = (hi - lo + kThreads) / kThreads;
        const int64_t v = lo + (int64_t)threadIdx.x * step;
        const int c = __syncthreads_count(v <= hi && tile_off[v] <= t);   // >= 1 (probe lo)
        const int64_t nlo = lo + (int64_t)(c - 1) * step;
        hi = min(hi, nlo + step - 1);
        lo = nlo;
    }
    return lo;
}

// a goes first in a merge (ties go to the first run).
template <typename F>
__device__ __forceinline__ bool first_le(const typename F::T &a, const typename F::T &b) {
    return !F::less(b, a);
}

// Compare-exchange: afterwards a <= b when up, a >= b otherwise.
template <typename F>
__device__ __forceinline__ void cx(typename F::T &a, typename F::T &b, bool up) {
    const bool sw = up ? F::less(b, a) : F::less(a, b);
    const typename F::T x = F::sel(sw, b, a), y = F::sel(sw, a, b);
    a = x;
    b = y;
}

// Bitonic network over a thread's kEpt registers. Written with template recursion so that every
// register index is a compile-time constant (a runtime partner index would put the array in
// scratch memory).
template <typename F, int K, int J>
__device__ __forceinline__ void bitonic_stage(typename F::T (&r)[kEpt]) {
#pragma unroll
    for (int i = 0; i < kEpt; ++i) {
        const int p = i ^ J;
        if (p > i)
            cx<F>(r[i], r[p], (i & K) == 0);
    }
    if constexpr (J > 1)
        bitonic_stage<F, K, J / 2>(r);
}

template <typename F, int K>
__device__ __forceinline__ void bitonic_level(typename F::T (&r)[kEpt]) {
    bitonic_stage<F, K, K / 2>(r);
    if constexpr (K < kEpt)
        bitonic_level<F, K * 2>(r);
}

template <typename F>
__device__ __forceinline__ void sort_regs(typename F::T (&r)[kEpt]) {
    bitonic_level<F, 2>(r);
}

// Outputs [d, d + kEpt) of merge(A, B), A = s[a_off, a_off + la), B = s[b_off, b_off + lb)
// (logical indices, padded in LDS). Outputs past la + lb are pad elements.
template <typename F>
__device__ __forceinline__ void merge_ept(const typename F::T *s, int a_off, int la, int b_off,
                                          int lb, int d, typename F::T (&r)[kEpt]) {
    typedef typename F::T T;
    int lo = d > lb ? d - lb : 0, hi = d < la ? d : la;
    while (lo < hi) {                      // smallest i with A[i] not among the first d outputs
        const int mid = (lo + hi) >> 1;
        if (first_le<F>(s[pidx(a_off + mid)], s[pidx(b_off + d - 1 - mid)]))
            lo = mid + 1;
        else
            hi = mid;
    }
    int ia = lo, ib = d - lo;
    T a = ia < la ? s[pidx(a_off + ia)] : F::pad();
    T b = ib < lb ? s[pidx(b_off + ib)] : F::pad();
#pragma unroll
    for (int m = 0; m < kEpt; ++m) {
        const bool take_a = ib >= lb || (ia < la && first_le<F>(a, b));
        r[m] = F::sel(take_a, a, b);
        ia += take_a;
        ib += !take_a;
        const bool ok = take_a ? ia < la : ib < lb;
        const T nx = ok ? s[pidx(take_a ? a_off + ia : b_off + ib)] : F::pad();
        a = F::sel(take_a, nx, a);
        b = F::sel(take_a, b, nx);
    }
}

template <typename F>
__device__ __forceinline__ void store_regs(typename F::T *s, const typename F::T (&r)[kEpt],
                                           int first, int n) {
#pragma unroll
    for (int m = 0; m < kEpt; ++m)
        if (first + m < n)
            s[pidx(first + m)] = r[m];
}

struct SortOut {
    int64_t limit;          // viewers with more records are copied through in input order
    int64_t total;
    const chunk_t *rows_in;
    int32_t row_chunks;
    int64_t *keys_out;
    chunk_t *rows_out;
    uint32_t *perm;         // [total]: input position of the record at each output position
};

// Copy the feature rows of n sorted records: record i's row goes from flat input position
// src(i) to flat output position dst(i), skipped where dst(i) < 0. 16-byte chunks in batches of U
// per thread, two batches in flight: the loads of the next batch are issued before the stores
// of the current one (vector-memory completions are counted in issue order, stores included, so
// a load issued after a store could only be waited for together with it). The sorted rows are
// not read again by this call: non-temporal stores keep them from evicting the lines of rows
// still to be gathered.
template <int U, typename Map>
__device__ __forceinline__ void copy_rows(int n, const SortOut &o, Map map) {
    const int row_chunks = o.row_chunks;
    const int n_chunks = n * row_chunks;
    // Chunk g of the thread's sequence (g = threadIdx.x + j * kThreads) is chunk q of record
    // rec; both advance by kThreads chunks without a division.
    const int drec = kThreads / row_chunks, dq = kThreads - drec * row_chunks;
    int rec = threadIdx.x / row_chunks, q = threadIdx.x - rec * row_chunks;
    auto load = [&](int g0, chunk_t (&c)[U], int64_t (&to)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int g = g0 + u * kThreads;
            to[u] = -1;
            if (g < n_chunks) {
                int64_t src, dst;
                map(rec, src, dst);
                if (dst >= 0) {
                    c[u] = o.rows_in[src * row_chunks + q];
                    to[u] = dst * row_chunks + q;
                }
            }
            rec += drec;
            q += dq;
            if (q >= row_chunks) {
                q -= row_chunks;
                ++rec;
            }
        }
    };
    auto store = [&](const chunk_t (&c)[U], const int64_t (&to)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (to[u] >= 0)
                __builtin_nontemporal_store(c[u], o.rows_out + to[u]);
    };
    chunk_t ca[U], cb[U];
    int64_t ta[U], tb[U];
    load(threadIdx.x, ca, ta);
    for (int g0 = threadIdx.x; g0 < n_chunks; g0 += 2 * U * kThreads) {
        load(g0 + U * kThreads, cb, tb);
        store(ca, ta);
        load(g0 + 2 * U * kThreads, ca, ta);
        store(cb, tb);
    }
}

// Records [base, base + n) go to the output unchanged, in input order (keys now, rows by the
// gather).
__device__ __forceinline__ void copy_through(const int64_t *__restrict__ keys, int64_t base, int n,
                                             const SortOut &o) {
    for (int i = threadIdx.x; i < n; i += kThreads) {
        o.keys_out[base + i] = keys[base + i];
        o.perm[base + i] = (uint32_t)(base + i);
    }
}

// ---- plan and key range --------------------------------------------------------------------

// Reduces the per-workgroup key ranges of range_kernel (n_slots pairs) into c.range = {min,
// max}; mt_off[v] = multi-tile tiles of viewers < v, for v in [0, B] (tiles of the element
// form's size); clears the pass counters. One workgroup.
__global__ __launch_bounds__(kThreads) void plan_kernel(const int64_t *off, int32_t B,
                                                        int64_t total, int64_t *mt_off,
                                                        const int64_t *slots, int n_slots,
                                                        Codec c, uint32_t *counters) {
    int64_t *range = const_cast<int64_t *>(c.range);
    __shared__ int64_t s[kThreads];
    __shared__ int64_t s_hi[kThreads];
    __shared__ int64_t carry;
    const int tid = threadIdx.x;
    if (tid < kMaxPasses)
        counters[tid] = 0;
    {
        int64_t lo = INT64_MAX, hi = INT64_MIN;
        for (int i = tid; i < n_slots; i += kThreads) {
            lo = min(lo, slots[2 * i]);
            hi = max(hi, slots[2 * i + 1]);
        }
        s[tid] = lo;
        s_hi[tid] = hi;
        lds_sync();
        for (int d = kThreads / 2; d > 0; d >>= 1) {
            if (tid < d) {
                s[tid] = min(s[tid], s[tid + d]);
                s_hi[tid] = max(s_hi[tid], s_hi[tid + d]);
            }
            lds_sync();
        }
        if (tid == 0) {
            range[0] = s[0];
            range[1] = s_hi[0];
            carry = 0;
        }
        lds_sync();
    }
    // The form from the reduced range in LDS (the range just written to global memory is not
    // read back here).
    const int tile = radix_tile(packs(s[0], s_hi[0], c.pbits));
    lds_sync();                                       // s is reused by the scan below
    for (int64_t b0 = 0; b0 <= B; b0 += kThreads) {
        const int64_t v = b0 + tid;
        int64_t n = 0;
        if (v < B) {
            int64_t kb, ke;
            segment(off, total, v, kb, ke);
            n = multi_tiles(ke - kb, tile);
        }
        s[tid] = n;
        lds_sync();
        for (int d = 1; d < kThreads; d <<= 1) {     // inclusive scan (Hillis-Steele)
            const int64_t x = tid >= d ? s[tid - d] : 0;
            lds_sync();
            s[tid] += x;
            lds_sync();
        }
        if (v <= B)
            mt_off[v] = carry + s[tid] - n;           // exclusive
        lds_sync();
        if (tid == kThreads - 1)
            carry += s[tid];
        lds_sync();
    }
}

// slots[2b], slots[2b + 1] = min and max of the keys workgroup b reads (a grid-stride slice of
// keys[0, total)); the plan kernel reduces the slots. No atomics and nothing to initialise.
constexpr int kRangeThreads = 256;
constexpr int kRangeUnroll = 4;

__global__ __launch_bounds__(kRangeThreads) void range_kernel(const int64_t *__restrict__ keys,
                                                              int64_t total, int64_t *slots) {
    __shared__ int64_t s_lo[kRangeThreads / 64], s_hi[kRangeThreads / 64];
    int64_t lo = INT64_MAX, hi = INT64_MIN;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < total;
         i0 += kRangeUnroll * stride) {
        int64_t k[kRangeUnroll];
#pragma unroll
        for (int u = 0; u < kRangeUnroll; ++u)
            k[u] = keys[min(i0 + u * stride, total - 1)];      // clamped: repeats change nothing
#pragma unroll
        for (int u = 0; u < kRangeUnroll; ++u) {
            lo = min(lo, k[u]);
            hi = max(hi, k[u]);
        }
    }
    for (int off = 32; off > 0; off >>= 1) {
        lo = min(lo, (int64_t)__shfl_down(lo, off));
        hi = max(hi, (int64_t)__shfl_down(hi, off));
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_lo[wave] = lo;
        s_hi[wave] = hi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int k = 1; k < kRangeThreads / 64; ++k) {
            lo = min(lo, s_lo[k]);
            hi = max(hi, s_hi[k]);
        }
        slots[2 * blockIdx.x] = lo;
        slots[2 * blockIdx.x + 1] = hi;
    }
}

// ---- small viewers: the whole viewer sorted in LDS -----------------------------------------

// Multi-tile context shared by the kernels below: mt_off from the plan, each tile's descriptor,
// the list's capacity (the workspace bound), the per-viewer digit histograms (row = the
// viewer's first tile in the list), the look-back status words (two sets, used by alternate
// passes) and the tile-claim counters (per viewer for the direct passes, one per pass for the
// looping ones).
struct Multi {
    const int64_t *mt_off;
    int64_t *desc;         // [mt_cap][4]: segment start, end and first list tile of each tile
    int64_t mt_cap;
    uint32_t *hist;        // [mt_cap][kMaxPasses][kRadix]
    uint64_t *status;      // [2][mt_cap][kRadix]
    uint32_t *counters;    // [kMaxPasses] tile claims of the looping passes
    uint32_t *vclaim;      // [mt_cap][kMaxPasses] tile claims per viewer (row = first tile)
};

template <typename F>
__device__ __forceinline__ void small_body(const F &fm, const Digits &dg, char *lds,
                                           const int64_t *__restrict__ keys, const int64_t *off,
                                           int32_t B, const Multi &mt, const SortOut &o) {
    typedef typename F::T T;
    T *s = reinterpret_cast<T *>(lds);
    const int tid = threadIdx.x;
    for (int64_t v = blockIdx.x; v < B; v += gridDim.x) {         // uniform per workgroup
        int64_t kb, ke;
        segment(off, o.total, v, kb, ke);
        const int n = (int)min<int64_t>(ke - kb, kTile + 1);
        if (n == 0)
            continue;
        if (n > kTile) {
            // A multi-tile viewer: clear its histogram before the histogram kernel adds to it.
            const int64_t row = mt.mt_off[v];
            if (ke - kb <= o.limit && row < mt.mt_cap)
                for (int j = tid; j < dg.P * kRadix; j += kThreads)
                    mt.hist[row * (kMaxPasses * kRadix) + j] = 0;
            continue;
        }
        if (n > o.limit) {                               // larger than the caller's bound
            copy_through(keys, kb, n, o);
            continue;
        }
#pragma unroll
        for (int m = 0; m < kEpt; ++m) {
            const int i = m * kThreads + tid;
            s[pidx(i)] = i < n ? fm.make(keys[kb + i], kb + i, kb) : F::pad();  // pads last
        }
        lds_sync();
        T r[kEpt];
#pragma unroll
        for (int m = 0; m < kEpt; ++m)
            r[m] = s[pidx(tid * kEpt + m)];
        sort_regs<F>(r);
        // Records sit at positions [0, n) and pads after them, so once the runs reach the power
        // of two p >= n the records are one sorted run; later rounds would only merge pads.
        int p = kEpt;
        while (p < n)
            p <<= 1;
        for (int L = kEpt; L < p; L <<= 1) {
            lds_sync();                                  // every thread has read s
            store_regs<F>(s, r, tid * kEpt, kTile);
            lds_sync();
            const int d = tid * kEpt;
            const int a_off = (d / (2 * L)) * (2 * L);
            merge_ept<F>(s, a_off, L, a_off + L, L, d - a_off, r);
        }
        lds_sync();
        store_regs<F>(s, r, tid * kEpt, kTile);
        lds_sync();
        for (int i = tid; i < n; i += kThreads) {
            const T x = s[pidx(i)];
            __builtin_nontemporal_store(fm.key(x), o.keys_out + kb + i);
            o.perm[kb + i] = (uint32_t)clampk(fm.src(x, kb), o.total - 1);
        }
        lds_sync();                                      // s is reused by the next viewer
    }
}

__global__ __launch_bounds__(kThreads) void small_kernel(const int64_t *__restrict__ keys,
                                                         const int64_t *off, int32_t B, Multi mt,
                                                         SortOut o, Codec c) {
    __shared__ __attribute__((aligned(16))) char lds[kLdsElems * sizeof(Wide::T)];
    if (B <= 0)
        return;
    const Digits dg = digits_of(c);
    int64_t kmin;
    if (use_packed(c, kmin))
        small_body(Packed{kmin, c.pbits}, dg, lds, keys, off, B, mt, o);
    else
        small_body(Wide{kmin}, dg, lds, keys, off, B, mt, o);
}

// ---- merge path (calls below kRadixMinRecords records) -------------------------------------
//
// Tiles of kTile records per viewer (tile_off: an exclusive scan of ceil(n_v / kTile)); a block
// sort per tile, then merge rounds within each viewer: runs of kTile << r records are merged
// pairwise, one output tile per workgroup, whose two merge-path split points are found by
// 64-ary searches (one wavefront each). A viewer's last pass (its block sort when it has one
// tile, else its last merge round) writes the sorted keys and copies each record's feature row
// from the input; earlier passes write elements to the two ping-pong arrays.

// The first n records of s (sorted) belong at flat positions [pos, pos + n) of the viewer that
// starts at kb. Either write the elements to dst, or, on a viewer's last pass, the keys and the
// rows they came from.
template <typename F>
__device__ __forceinline__ void emit(const F &fm, const typename F::T *s, int n, int64_t pos,
                                     int64_t kb, typename F::T *__restrict__ dst, bool last,
                                     const SortOut &o) {
    const int tid = threadIdx.x;
    if (!last) {
        for (int i = tid; i < n; i += kThreads)
            dst[pos + i] = s[pidx(i)];
        return;
    }
    // The sorted keys and rows are not read again by this call: non-temporal stores keep them
    // from evicting the lines of rows still to be gathered.
    for (int i = tid; i < n; i += kThreads)
        __builtin_nontemporal_store(fm.key(s[pidx(i)]), o.keys_out + pos + i);
    constexpr int U = 8;
    const int row_chunks = o.row_chunks;
    const int n_chunks = n * row_chunks;
    for (int g0 = tid; g0 < n_chunks; g0 += U * kThreads) {
        chunk_t c[U];
        int64_t dst_i[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int g = g0 + u * kThreads;
            dst_i[u] = -1;
            if (g < n_chunks) {
                const int rec = g / row_chunks;
                const int q = g - rec * row_chunks;
                const int64_t f = clampk(fm.src(s[pidx(rec)], kb), o.total - 1);
                c[u] = o.rows_in[f * row_chunks + q];
                dst_i[u] = (pos + rec) * row_chunks + q;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (dst_i[u] >= 0)
                __builtin_nontemporal_store(c[u], o.rows_out + dst_i[u]);
    }
}

// tile_off[v] = sum of tiles of viewers < v, for v in [0, B]. One workgroup. Also reduces the
// per-workgroup key ranges of range_kernel (n_slots pairs) into range = {min, max}.
__global__ __launch_bounds__(kThreads) void merge_plan_kernel(const int64_t *off, int32_t B,
                                                        int64_t total, int64_t *tile_off,
                                                        const int64_t *slots, int n_slots,
                                                        int64_t *range) {
    __shared__ int64_t s[kThreads];
    __shared__ int64_t s_hi[kThreads];
    __shared__ int64_t carry;
    const int tid = threadIdx.x;
    {
        int64_t lo = INT64_MAX, hi = INT64_MIN;
        for (int i = tid; i < n_slots; i += kThreads) {
            lo = min(lo, slots[2 * i]);
            hi = max(hi, slots[2 * i + 1]);
        }
        s[tid] = lo;
        s_hi[tid] = hi;
        lds_sync();
        for (int d = kThreads / 2; d > 0; d >>= 1) {
            if (tid < d) {
                s[tid] = min(s[tid], s[tid + d]);
                s_hi[tid] = max(s_hi[tid], s_hi[tid + d]);
            }
            lds_sync();
        }
        if (tid == 0) {
            range[0] = s[0];
            range[1] = s_hi[0];
            carry = 0;
        }
        lds_sync();
    }
    for (int64_t b0 = 0; b0 <= B; b0 += kThreads) {
        const int64_t v = b0 + tid;
        int64_t n = 0;
        if (v < B) {
            int64_t kb, ke;
            segment(off, total, v, kb, ke);
            n = tiles_of(ke - kb);
        }
        s[tid] = n;
        lds_sync();
        for (int d = 1; d < kThreads; d <<= 1) {     // inclusive scan (Hillis-Steele)
            const int64_t x = tid >= d ? s[tid - d] : 0;
            lds_sync();
            s[tid] += x;
            lds_sync();
        }
        if (v <= B)
            tile_off[v] = carry + s[tid] - n;         // exclusive
        lds_sync();
        if (tid == kThreads - 1)
            carry += s[tid];
        lds_sync();
    }
}

// Records [base, base + n) go to the output unchanged (keys and rows, in input order).
__device__ __forceinline__ void copy_through_rows(const int64_t *__restrict__ keys, int64_t base, int n,
                                             const SortOut &o) {
    for (int i = threadIdx.x; i < n; i += kThreads)
        o.keys_out[base + i] = keys[base + i];
    const int64_t c0 = base * o.row_chunks;
    const int n_chunks = n * o.row_chunks;
    for (int g = threadIdx.x; g < n_chunks; g += kThreads)
        o.rows_out[c0 + g] = o.rows_in[c0 + g];
}

template <typename F>
__device__ __forceinline__ void block_sort_body(const F &fm, char *lds,
                                                const int64_t *__restrict__ keys,
                                                const int64_t *off, int32_t B,
                                                const int64_t *tile_off, void *out_v,
                                                const SortOut &o) {
    typedef typename F::T T;
    T *s = reinterpret_cast<T *>(lds);
    T *out = static_cast<T *>(out_v);
    const int tid = threadIdx.x;
    const int64_t n_tiles = tile_off[B];
    for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {   // uniform per workgroup
        const int64_t v = owner(tile_off, B, t);
        int64_t kb, ke;
        segment(off, o.total, v, kb, ke);
        const int64_t base = kb + (t - tile_off[v]) * kTile;
        const int n = (int)(min<int64_t>(base + kTile, ke) - base);
        const bool last = tile_off[v + 1] - tile_off[v] == 1;
        if (ke - kb > o.limit) {                         // larger than the caller's bound
            copy_through_rows(keys, base, n, o);
            continue;
        }
#pragma unroll
        for (int m = 0; m < kEpt; ++m) {
            const int i = m * kThreads + tid;
            s[pidx(i)] = i < n ? fm.make(keys[base + i], base + i, kb) : F::pad();  // pads last
        }
        lds_sync();
        T r[kEpt];
#pragma unroll
        for (int m = 0; m < kEpt; ++m)
            r[m] = s[pidx(tid * kEpt + m)];
        sort_regs<F>(r);
        // Records sit at positions [0, n) and pads after them, so once the runs reach the power
        // of two p >= n the records are one sorted run; later rounds would only merge pads.
        int p = kEpt;
        while (p < n)
            p <<= 1;
        for (int L = kEpt; L < p; L <<= 1) {
            lds_sync();                                  // every thread has read s
            store_regs<F>(s, r, tid * kEpt, kTile);
            lds_sync();
            const int d = tid * kEpt;
            const int a_off = (d / (2 * L)) * (2 * L);
            merge_ept<F>(s, a_off, L, a_off + L, L, d - a_off, r);
        }
        lds_sync();
        store_regs<F>(s, r, tid * kEpt, kTile);
        lds_sync();
        emit<F>(fm, s, n, base, kb, out, last, o);
        lds_sync();                                      // s is reused by the next tile
    }
}

__global__ __launch_bounds__(kThreads) void block_sort_kernel(const int64_t *__restrict__ keys,
                                                              const int64_t *off, int32_t B,
                                                              const int64_t *tile_off,
                                                              void *out, SortOut o, Codec c) {
    __shared__ __attribute__((aligned(16))) char lds[kLdsElems * sizeof(Wide::T)];
    if (B <= 0)
        return;
    int64_t kmin;
    if (use_packed(c, kmin))
        block_sort_body(Packed{kmin, c.pbits}, lds, keys, off, B, tile_off, out, o);
    else
        block_sort_body(Wide{kmin}, lds, keys, off, B, tile_off, out, o);
}

// Merge-path split: the number of A elements among the first d outputs of merge(A, B), i.e.
// the smallest i in [lo, hi] such that A[i] is not among them. Run by all 64 lanes of one
// wavefront (64 probes per round); returns the same value in every lane.
template <typename F>
__device__ int64_t split64(const typename F::T *A, int64_t la, const typename F::T *B, int64_t lb,
                           int64_t d) {
    int64_t lo = d > lb ? d - lb : 0;
    int64_t hi = d < la ? d : la;
    const int lane = threadIdx.x & 63;
    while (hi > lo) {
        const int64_t n = hi - lo;
        const int64_t step = (n + 63) / 64;
        const int64_t m = lo + lane * step;
        bool in_out = false;                     // A[m] is among the first d outputs
        if (m < hi)
            in_out = first_le<F>(A[m], B[d - 1 - m]);
        const uint64_t ballot = __ballot(m < hi && !in_out);
        if (step == 1)
            return ballot ? lo + __builtin_ctzll(ballot) : hi;   // first false, else hi
        if (ballot == 0) {
            // Every probe in range was true: the answer lies past the last one in range.
            const int64_t last = min<int64_t>(63, (n - 1) / step);
            lo = lo + last * step + 1;
        } else {
            const int first = __builtin_ctzll(ballot);
            const int64_t new_hi = lo + first * step;
            lo = first == 0 ? lo : lo + (first - 1) * step + 1;
            hi = new_hi;
        }
    }
    return lo;
}

template <typename F>
__device__ __forceinline__ void merge_body(const F &fm, char *lds, int64_t *s_split,
                                           const void *src_v, void *dst_v, const int64_t *off,
                                           int32_t B, const int64_t *tile_off, int r,
                                           const SortOut &o) {
    typedef typename F::T T;
    T *s = reinterpret_cast<T *>(lds);
    const T *src = static_cast<const T *>(src_v);
    T *dst = static_cast<T *>(dst_v);
    const int tid = threadIdx.x;
    const int64_t n_tiles = tile_off[B];
    for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {   // uniform per workgroup
        const int64_t v = owner(tile_off, B, t);
        const int64_t nt = tile_off[v + 1] - tile_off[v];
        if (((int64_t)1 << r) >= nt)
            continue;                                    // this viewer is already sorted
        const bool last = r == rounds_of(nt) - 1;
        int64_t kb, ke;
        segment(off, o.total, v, kb, ke);
        if (ke - kb > o.limit)
            continue;                                    // copied through by the block sort
        const int64_t n_seg = ke - kb;
        const int64_t run = (int64_t)kTile << r;
        const int64_t out0 = (t - tile_off[v]) * kTile;  // position within the viewer
        const int64_t a0 = (out0 / (2 * run)) * 2 * run;
        const int64_t la = min(run, n_seg - a0);
        const int64_t b0 = a0 + la;
        const int64_t lb = max<int64_t>(0, min(run, n_seg - b0));
        const int64_t d0 = out0 - a0;
        const int64_t d1 = min<int64_t>(d0 + kTile, la + lb);
        const T *A = src + kb + a0;
        const T *Bv = src + kb + b0;
        if (tid < 128) {                                 // wavefront 0: d0, wavefront 1: d1
            const int64_t i = split64<F>(A, la, Bv, lb, tid < 64 ? d0 : d1);
            if ((tid & 63) == 0)
                s_split[tid >> 6] = i;
        }
        lds_sync();
        const int64_t i0 = s_split[0], i1 = s_split[1];
        const int64_t j0 = d0 - i0;
        // For sorted runs i0 <= i1 and j0 <= j1; the clamp keeps every access inside the runs
        // even when malformed offsets made two viewers overlap.
        const int n = (int)(d1 - d0);
        const int na = (int)min<int64_t>(max<int64_t>(i1 - i0, 0), n), nb = n - na;
        // A[i0, i0 + na) then B[j0, j0 + nb) side by side in LDS.
#pragma unroll 4
        for (int i = tid; i < n; i += kThreads)
            s[pidx(i)] = i < na ? A[i0 + i] : Bv[j0 + (i - na)];
        lds_sync();
        T rr[kEpt];
        const int d = tid * kEpt;
        if (d < n)
            merge_ept<F>(s, 0, na, na, nb, d, rr);
        lds_sync();
        if (d < n)
            store_regs<F>(s, rr, d, n);
        lds_sync();
        emit<F>(fm, s, n, kb + a0 + d0, kb, dst, last, o);
        lds_sync();                                      // s and s_split are reused
    }
}

// Round r: within every viewer with more than 2^r tiles, merge runs of kTile << r records
// pairwise from src into dst (a run without a partner is copied).
__global__ __launch_bounds__(kThreads) void merge_kernel(const void *src, void *dst,
                                                         const int64_t *off, int32_t B,
                                                         const int64_t *tile_off, int r,
                                                         SortOut o, Codec c) {
    __shared__ __attribute__((aligned(16))) char lds[kLdsElems * sizeof(Wide::T)];
    __shared__ int64_t s_split[2];
    if (B <= 0)
        return;
    int64_t kmin;
    if (use_packed(c, kmin))
        merge_body(Packed{kmin, c.pbits}, lds, s_split, src, dst, off, B, tile_off, r, o);
    else
        merge_body(Wide{kmin}, lds, s_split, src, dst, off, B, tile_off, r, o);
}

// ---- multi-tile viewers: digit histograms ----------------------------------------------------

// Tile t of the multi-tile list: its viewer v, the viewer's segment and first list tile, and
// the tile's records [base, base + n).
struct TileAt {
    int64_t v, kb, ke, t0, base;
    int n;
};

__device__ __forceinline__ TileAt tile_at(const int64_t *off, int32_t B, const Multi &mt,
                                          int64_t total, int64_t t, int tile) {
    TileAt a;
    a.v = owner(mt.mt_off, B, t);
    segment(off, total, a.v, a.kb, a.ke);
    a.t0 = mt.mt_off[a.v];
    a.base = a.kb + (t - a.t0) * tile;
    a.n = (int)clampk(a.ke - a.base, tile);
    return a;
}

// Counts of every digit value of every pass over each multi-tile viewer's records, added into
// the viewer's histogram (cleared by the small-viewer kernel). Also clears the tile's
// look-back status for the first pass, and copies the tiles of viewers above the caller's
// bound through.
__global__ __launch_bounds__(kThreads) void hist_kernel(const int64_t *__restrict__ keys,
                                                        const int64_t *off, int32_t B, Multi mt,
                                                        SortOut o, Codec c) {
    __shared__ uint32_t s_h[kMaxPasses * kRadix];
    if (B <= 0)
        return;
    const int tid = threadIdx.x;
    const Digits dg = digits_of(c);
    int64_t kmin_s;
    const int tile = radix_tile(use_packed(c, kmin_s));
    const uint64_t kmin = (uint64_t)kmin_s;
    const int64_t n_mt = min(mt.mt_off[B], mt.mt_cap);
    for (int64_t t = blockIdx.x; t < n_mt; t += gridDim.x) {     // uniform per workgroup
        const TileAt a = tile_at(off, B, mt, o.total, t, tile);
        if (tid < 3)
            mt.desc[t * 4 + tid] = tid == 0 ? a.kb : (tid == 1 ? a.ke : a.t0);
        if (t == a.t0 && tid < kMaxPasses)
            mt.vclaim[t * kMaxPasses + tid] = 0;         // the viewer's claim counters
        if (a.ke - a.kb > o.limit) {
            copy_through(keys, a.base, a.n, o);
            continue;
        }
        for (int j = tid; j < dg.P * kRadix; j += kThreads)
            s_h[j] = 0;
        if (tid < kRadix)
            mt.status[t * kRadix + tid] = 0;
        lds_sync();
        for (int i = tid; i < a.n; i += kThreads) {
            const uint64_t u = (uint64_t)keys[a.base + i] - kmin;
            for (int p = 0; p < dg.P; ++p)
                atomicAdd(&s_h[p * kRadix + ((u >> (p * dg.D)) & dg.mask)], 1u);
        }
        lds_sync();
        uint32_t *row = mt.hist + a.t0 * (kMaxPasses * kRadix);
        for (int j = tid; j < dg.P * kRadix; j += kThreads) {
            const uint32_t n = s_h[j];
            if (n)
                atomicAdd(row + j, n);
        }
        lds_sync();                                      // s_h is reused by the next tile
    }
}

// ---- multi-tile viewers: one digit pass ------------------------------------------------------

// Look-back status word of one tile and digit value: flag in the top two bits (0 = not yet
// published, kAgg = the tile's own count, kInc = count of this and every earlier tile of the
// viewer), the count below them.
constexpr uint64_t kAgg = (uint64_t)1 << 62;
constexpr uint64_t kInc = (uint64_t)2 << 62;
constexpr uint64_t kCountMask = kAgg - 1;
// Bound on the polls of one status word (each poll is a device-scope load, about a
// microsecond). A tile waits only for earlier tiles of its viewer, each held by a running
// workgroup that publishes its own counts before it looks back, so a wait lasts about one
// tile's ranking and the bound is never reached; it keeps every wave's exit certain.
constexpr int kMaxPolls = 1 << 13;

__device__ __forceinline__ void put_status(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t get_status(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Records of digit value d in tiles first .. k of one viewer (k >= first; tile `first`
// publishes kInc directly): walk back from k, adding published counts, until an inclusive one.
// The words of kLookBatch tiles are loaded at once, so a walk over many tiles that have only
// published their own counts costs one load latency per batch rather than per tile.
constexpr int kLookBatch = 8;

__device__ int64_t look_back(const uint64_t *st, int64_t first, int64_t k, int d) {
    int64_t sum = 0;
    int polls = 0;
    bool done = k < first;
    while (!done) {
        uint64_t w[kLookBatch];
#pragma unroll
        for (int j = 0; j < kLookBatch; ++j)
            w[j] = get_status(st + max(k - j, first) * kRadix + d);
#pragma unroll
        for (int j = 0; j < kLookBatch; ++j) {
            if (done)
                break;
            uint64_t x = w[j];
            while ((x & ~kCountMask) == 0 && polls < kMaxPolls) {
                ++polls;
                __builtin_amdgcn_s_sleep(1);
                x = get_status(st + max(k - j, first) * kRadix + d);
            }
            const uint64_t flag = x & ~kCountMask;
            sum += (int64_t)(x & kCountMask);
            // Tile `first` (reached at the latest when k - j == first) is inclusive; a word
            // still unpublished after the poll bound ends the walk.
            done = flag != kAgg;
        }
        k -= kLookBatch;
    }
    return sum;
}

// Exclusive prefix sum of x over threads [0, kRadix) (other threads pass 0 and get their
// wavefront's prefix). Every thread calls it; s_w holds kRadix / 64 partial sums.
__device__ __forceinline__ int64_t radix_excl_scan(int64_t x, int64_t *s_w) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    int64_t inc = x;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_up(inc, d);
        if (lane >= d)
            inc += y;
    }
    if (lane == 63 && w < kRadix / 64)
        s_w[w] = inc;
    lds_sync();
    int64_t base = 0;
#pragma unroll
    for (int k = 0; k < kRadix / 64; ++k)
        base += k < w ? s_w[k] : 0;
    return base + inc - x;
}

static_assert(kRadix == kThreads, "one thread per digit value");

struct PassShared {
    uint16_t cnt[kWaves][kRadix];   // per wavefront: running count, then its exclusive prefix
    uint32_t go[kRadix];            // viewer position of tile-sorted record i: go[digit] + i
                                    // (modulo 2^32; viewers hold fewer than 2^32 records)
    int32_t start[kRadix];          // first tile-sorted index of each digit value
    int64_t scan_a[kRadix / 64], scan_b[kRadix / 64];
    int64_t tile;
    int64_t desc[3];                // the tile's segment start and end, and its viewer's first tile
};

// Digit pass p over tile t of the multi-tile list (called by the whole workgroup), whose
// descriptor is in sh.desc.
template <typename F>
__device__ __forceinline__ void pass_tile(const F &fm, const Digits &dg, int p, char *lds,
                                          PassShared &sh, const int64_t *__restrict__ keys,
                                          const void *src_v, void *dst_v, const Multi &mt,
                                          const SortOut &o, int64_t t) {
    typedef typename F::T T;
    constexpr int E = F::kRadixEpt;
    T *s = reinterpret_cast<T *>(lds);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const bool last = p == dg.P - 1;
    const int shift = p * dg.D;
    uint64_t *st = mt.status + (int64_t)(p & 1) * mt.mt_cap * kRadix;
    uint64_t *st_next = mt.status + (int64_t)((p + 1) & 1) * mt.mt_cap * kRadix;
    const uint64_t below_me = (((uint64_t)1) << lane) - 1;
    {
        // The tile's segment, from the descriptor the histogram kernel wrote.
        TileAt a;
        a.kb = sh.desc[0];
        a.ke = sh.desc[1];
        a.t0 = sh.desc[2];
        a.base = a.kb + (t - a.t0) * (E * kThreads);
        a.n = (int)clampk(a.ke - a.base, E * kThreads);
        if (a.ke - a.kb > o.limit)
            return;                                      // copied through by hist_kernel
        const uint32_t nv = (uint32_t)(a.ke - a.kb);
        if (tid < kRadix)
            st_next[t * kRadix + tid] = 0;               // for the next pass, which starts later

        // Records of wavefront w: [w * 64 * E, (w + 1) * 64 * E), E rounds of 64, so that
        // (wavefront, round, lane) is the input order.
        T e[E];
        {
            const int64_t *kin = keys + a.base;
            const T *in = static_cast<const T *>(src_v) + a.base;
#pragma unroll
            for (int m = 0; m < E; ++m) {
                const int i = (w * E + m) * 64 + lane;
                if (p == 0)
                    e[m] = i < a.n ? fm.make(kin[i], a.base + i, a.kb) : F::pad();
                else
                    e[m] = i < a.n ? in[i] : F::pad();
            }
        }
        // Per wavefront: its digit counts, and one 64-bit lane-mask word per digit value (in the
        // tile's LDS area, free until the scatter).
        uint64_t *flags = reinterpret_cast<uint64_t *>(lds) + w * kRadix;
        for (int j = lane; j < kRadix; j += 64) {
            sh.cnt[w][j] = 0;
            flags[j] = 0;
        }
        // The viewer's records of each smaller digit value: where the digit's records start.
        const uint32_t h =
            tid < kRadix ? mt.hist[(a.t0 * kMaxPasses + p) * kRadix + tid] : 0u;
        const int64_t vstart = radix_excl_scan(h, sh.scan_a);    // has a barrier

        // Rank within the wavefront: records of equal digit before this one in earlier rounds
        // (the wavefront's running count) and in this round (lower lanes). The lanes of a round
        // OR their bits into the wavefront's word for their digit and read it back: the lanes
        // holding that digit (the wavefront's LDS accesses complete in order, so every OR of
        // the round precedes every read). The lowest lane of each digit group then advances
        // the count and clears the word, after every lane of the group has read both.
        // rd[m] = (rank << 16) | digit: one register per record, pinned here so that the
        // compiler does not keep the masks and partial counts it derives from alive until the
        // scatter below.
        uint32_t rd[E];
#pragma unroll
        for (int m = 0; m < E; ++m) {
            const bool valid = (w * E + m) * 64 + lane < a.n;
            const uint32_t d = fm.digit(e[m], shift, dg.mask);
            uint64_t peers = 0;
            uint32_t c = 0;
            if (valid) {
                __hip_atomic_fetch_or(&flags[d], ((uint64_t)1) << lane, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_WAVEFRONT);
                peers = __hip_atomic_load(&flags[d], __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_WAVEFRONT);
                c = sh.cnt[w][d];
            }
            const uint32_t before = (uint32_t)__popcll(peers & below_me);
            if (valid && before == 0) {
                sh.cnt[w][d] = (uint16_t)(c + (uint32_t)__popcll(peers));
                __hip_atomic_store(&flags[d], (uint64_t)0, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_WAVEFRONT);
            }
            uint32_t x = ((c + before) << 16) | d;
            asm volatile("" : "+v"(x));
            rd[m] = x;
        }
        lds_sync();
        uint32_t tot = 0;
        if (tid < kRadix) {
            for (int k = 0; k < kWaves; ++k) {
                const uint32_t c = sh.cnt[k][tid];
                sh.cnt[k][tid] = (uint16_t)tot;
                tot += c;
            }
        }
        const int64_t tstart = radix_excl_scan(tot, sh.scan_b);  // has a barrier
        if (tid < kRadix) {
            uint64_t *mine = st + t * kRadix + tid;
            int64_t before_tile = 0;
            if (t == a.t0) {
                put_status(mine, kInc | tot);
            } else {
                put_status(mine, kAgg | tot);
                before_tile = look_back(st, a.t0, t - 1, tid);
                put_status(mine, kInc | (uint64_t)(before_tile + tot));
            }
            sh.start[tid] = (int32_t)tstart;
            sh.go[tid] = (uint32_t)(vstart + before_tile - tstart);
        }
        lds_sync();
#pragma unroll
        for (int m = 0; m < E; ++m) {
            if ((w * E + m) * 64 + lane < a.n) {
                const uint32_t d = rd[m] & 0xFFFFu;
                s[sh.start[d] + sh.cnt[w][d] + (rd[m] >> 16)] = e[m];
            }
        }
        lds_sync();

        // Tile-sorted record i goes to viewer position go[digit] + i; records of one digit
        // value are consecutive there. Positions outside the viewer (only for malformed offsets)
        // are skipped, so every write stays inside the buffers.
        if (!last) {
            T *out = static_cast<T *>(dst_v) + a.kb;
            for (int i = tid; i < a.n; i += kThreads) {
                const T x = s[i];
                const uint32_t to = sh.go[fm.digit(x, shift, dg.mask)] + (uint32_t)i;
                if (to < nv)
                    out[to] = x;
            }
            return;
        }
        // Last digit: the sorted keys and, for the gather, each output position's input position.
        for (int i = tid; i < a.n; i += kThreads) {
            const T x = s[i];
            const uint32_t to = sh.go[fm.digit(x, shift, dg.mask)] + (uint32_t)i;
            if (to < nv) {
                __builtin_nontemporal_store(fm.key(x), o.keys_out + a.kb + to);
                o.perm[a.kb + to] = (uint32_t)clampk(fm.src(x, a.kb), o.total - 1);
            }
        }
    }
}

// Tiles of digit pass p, taken in claim order. LOOP = false: one tile per workgroup, the first
// n_mt workgroups claiming the n_mt tiles (from per-viewer counters, so that only a viewer's
// workgroups contend) and the rest of the grid (sized for the list's capacity) leaving without
// a claim. LOOP = true: a smaller grid whose workgroups claim tiles from one counter until none
// is left (a workgroup claims its next tile only after publishing the last one).
template <typename F, bool LOOP>
__device__ __forceinline__ void pass_body(const F &fm, const Digits &dg, int p, char *lds,
                                          PassShared &sh, const int64_t *__restrict__ keys,
                                          const void *src_v, void *dst_v, const int64_t *off,
                                          int32_t B, const Multi &mt, const SortOut &o) {
    const int64_t n_mt = min(mt.mt_off[B], mt.mt_cap);
    auto fetch_desc = [&](int64_t t) {
        const int64_t *d = mt.desc + t * 4;
        sh.desc[0] = d[0];
        sh.desc[1] = d[1];
        sh.desc[2] = d[2];
    };
    if constexpr (!LOOP) {
        if (threadIdx.x == 0) {
            // Workgroup b < n_mt takes a tile of the viewer that tile b belongs to, in that
            // viewer's claim order: as many workgroups as the viewer has tiles claim from its
            // counter, and every tile shares the viewer's descriptor.
            int64_t t = n_mt;
            if (blockIdx.x < n_mt) {
                fetch_desc(blockIdx.x);
                const int64_t t0 = sh.desc[2];
                t = t0 + (int64_t)atomicAdd(&mt.vclaim[t0 * kMaxPasses + p], 1u);
            }
            sh.tile = t;
        }
        lds_sync();
        const int64_t t = sh.tile;
        if (t < n_mt)                                    // uniform
            pass_tile(fm, dg, p, lds, sh, keys, src_v, dst_v, mt, o, t);
    } else {
        for (;;) {
            lds_sync();                                  // every thread is done with sh and lds
            if (threadIdx.x == 0) {
                const int64_t t = (int64_t)atomicAdd(&mt.counters[p], 1u);
                if (t < n_mt)
                    fetch_desc(t);
                sh.tile = t;
            }
            lds_sync();
            const int64_t t = sh.tile;
            if (t >= n_mt)
                break;                                   // uniform
            pass_tile(fm, dg, p, lds, sh, keys, src_v, dst_v, mt, o, t);
        }
    }
}

// Pass p of the call's P digit passes (launches for p >= P return at once). Pass 0 reads the
// input keys; later passes read the previous pass's elements (ping-pong buffers).
template <bool LOOP>
__global__ __launch_bounds__(kThreads, 4) void pass_kernel(const int64_t *__restrict__ keys,
                                                        const void *src, void *dst,
                                                        const int64_t *off, int32_t B, Multi mt,
                                                        int p, SortOut o, Codec c) {
    __shared__ __attribute__((aligned(16))) char lds[Wide::kRadixEpt * kThreads * sizeof(Wide::T)];
    __shared__ PassShared sh;
    if (B <= 0)
        return;
    const Digits dg = digits_of(c);
    if (p >= dg.P)
        return;
    int64_t kmin;
    if (use_packed(c, kmin))
        pass_body<Packed, LOOP>(Packed{kmin, c.pbits}, dg, p, lds, sh, keys, src, dst, off, B,
                                mt, o);
    else
        pass_body<Wide, LOOP>(Wide{kmin}, dg, p, lds, sh, keys, src, dst, off, B, mt, o);
}

// Rows of the sorted output: rows_out[i] = rows_in[perm[i]] for i in [0, total). Every output
// position is written by exactly one of the kernels above (the small-viewer sort, the copy
// through, or the last digit pass), so the gather runs over the whole array: kThreads rows per
// workgroup, their input positions staged in LDS.
__global__ __launch_bounds__(kThreads) void gather_kernel(SortOut o) {
    __shared__ uint32_t s_perm[kThreads];
    for (int64_t r0 = (int64_t)blockIdx.x * kThreads; r0 < o.total;
         r0 += (int64_t)gridDim.x * kThreads) {                  // uniform per workgroup
        const int n = (int)min<int64_t>(kThreads, o.total - r0);
        lds_sync();                                  // the previous rows' readers are done
        if ((int)threadIdx.x < n)
            s_perm[threadIdx.x] = min<uint32_t>(o.perm[r0 + threadIdx.x], (uint32_t)(o.total - 1));
        lds_sync();
        copy_rows<4>(n, o, [&](int rec, int64_t &from, int64_t &to) {
            from = (int64_t)s_perm[rec];
            to = r0 + rec;
        });
    }
}

constexpr int64_t round_up(int64_t x) { return (x + 255) & ~int64_t(255); }

constexpr int kRangeSlots = 1024;   // range_kernel workgroups at most

// Capacity of the multi-tile list: a viewer with n > kTile records has ceil(n / t) <= 2n / kTile
// tiles of t >= kTile records, so valid offsets give at most 2 * total / kTile.
constexpr int64_t multi_cap(int64_t total) { return 2 * total / kTile + 1; }

// Workspace layout: two ping-pong element arrays, mt_off, the key range and pass counters
// (256 bytes), the range kernel's per-workgroup slots, the digit histograms, the look-back
// status words, the tile descriptors, the per-viewer claim counters and the gather's input
// positions.
struct Layout {
    int64_t buf, mt_off, range, slots, hist, status, desc, vclaim, perm, bytes;
};

constexpr Layout layout_of(int64_t total, int64_t n_viewers) {
    const int64_t buf = round_up(total * (int64_t)sizeof(Wide::T));
    const int64_t cap = multi_cap(total);
    Layout l{};
    l.buf = buf;
    l.mt_off = 2 * buf;
    l.range = l.mt_off + round_up((n_viewers + 1) * 8);
    l.slots = l.range + 256;
    l.hist = l.slots + round_up(2 * kRangeSlots * 8);
    l.status = l.hist + round_up(cap * kMaxPasses * kRadix * 4);
    l.desc = l.status + round_up(2 * cap * kRadix * 8);
    l.vclaim = l.desc + round_up(cap * 4 * 8);
    l.perm = l.vclaim + round_up(cap * kMaxPasses * 4);
    l.bytes = l.perm + round_up(total * 4);
    return l;
}

// Fixed device scratch of the allocation-free sort (cc_sort_affinity_noalloc): the workspace of
// the largest call it accepts. One copy per device, resolved once per device below; in host
// code `scratch` names a host-side stand-in, so only the resolved address is ever passed on.
constexpr int64_t kScratchBytes = layout_of(kSortScratchRecords, kSortScratchViewers).bytes;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

}  // namespace

int64_t sort_workspace_bytes(int64_t total, int32_t n_viewers) {
    // Counts the sort rejects (total >= 2^32) need no workspace; this also keeps the products
    // below far from overflow.
    if (total <= 0 || n_viewers <= 0 || total >= ((int64_t)1 << 32))
        return 0;
    return layout_of(total, n_viewers).bytes;
}

hipError_t sort_scratch(int device, void **ptr) {
    static std::mutex mu;
    static void *addr[kMaxScratchDevices] = {};
    if (device < 0 || device >= kMaxScratchDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[device]) {
        // The caller has made `device` current: the symbol resolves to that device's copy.
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        addr[device] = p;
    }
    *ptr = addr[device];
    return hipSuccess;
}

hipError_t launch_sort(int32_t n_viewers, const int64_t *key_offsets, const int64_t *keys_in,
                       const void *rows_in, int32_t row_bytes, int64_t total, int64_t max_keys,
                       int64_t *keys_out, void *rows_out, void *workspace, int32_t method,
                       int32_t key_bits, hipStream_t stream) {
    if (total <= 0 || n_viewers <= 0)
        return hipSuccess;
    if (method == kSortAuto)
        method = total >= kSortRadixMinRecords ? kSortRadix : kSortMerge;
    uint8_t *w = static_cast<uint8_t *>(workspace);
    const Layout l = layout_of(total, n_viewers);
    void *buf0 = w;
    void *buf1 = w + l.buf;
    int64_t *mt_off = reinterpret_cast<int64_t *>(w + l.mt_off);   // tile_off on the merge path
    int64_t *range = reinterpret_cast<int64_t *>(w + l.range);
    uint32_t *counters = reinterpret_cast<uint32_t *>(w + l.range + 64);
    int64_t *slots = reinterpret_cast<int64_t *>(w + l.slots);
    const int64_t largest = max_keys > 0 ? (max_keys < total ? max_keys : total) : total;
    // Position bits of a packed element: enough for the largest viewer.
    int32_t pbits = 1;
    while (((int64_t)1 << pbits) < largest)
        ++pbits;
    // Digit passes to launch: enough for a key span of key_bits bits (64 when unknown).
    const int bits = key_bits > 0 && key_bits < 64 ? key_bits : 64;
    const int passes = (bits + kDigitBits - 1) / kDigitBits;
    const Codec c{range, pbits, passes < kMaxPasses ? passes : kMaxPasses};
    const SortOut o{largest, total, static_cast<const chunk_t *>(rows_in), row_bytes / 16,
                    keys_out, static_cast<chunk_t *>(rows_out),
                    reinterpret_cast<uint32_t *>(w + l.perm)};
    int64_t n_slots = (total + kRangeThreads * kRangeUnroll - 1) / (kRangeThreads * kRangeUnroll);
    if (n_slots > kRangeSlots)
        n_slots = kRangeSlots;
    hipLaunchKernelGGL(range_kernel, dim3((unsigned)n_slots), dim3(kRangeThreads), 0, stream,
                       keys_in, total, slots);
    hipError_t e = hipGetLastError();

    if (method == kSortMerge) {
        // Upper bound on tiles (every viewer adds at most one partial tile); larger counts are
        // covered by the kernels' grid-stride loops. Merge rounds from the largest viewer.
        int64_t grid = (total + kTile - 1) / kTile + n_viewers;
        if (grid > (1 << 20))
            grid = 1 << 20;
        const int64_t per_viewer = (largest + kTile - 1) / kTile;
        int rounds = 0;
        while (((int64_t)1 << rounds) < per_viewer)
            ++rounds;
        if (e == hipSuccess) {
            hipLaunchKernelGGL(merge_plan_kernel, dim3(1), dim3(kThreads), 0, stream, key_offsets,
                               n_viewers, total, mt_off, slots, (int)n_slots, range);
            e = hipGetLastError();
        }
        if (e == hipSuccess) {
            hipLaunchKernelGGL(block_sort_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream,
                               keys_in, key_offsets, n_viewers, mt_off, buf0, o, c);
            e = hipGetLastError();
        }
        for (int r = 0; e == hipSuccess && r < rounds; ++r) {
            const void *src = (r & 1) ? buf1 : buf0;
            void *dst = (r & 1) ? buf0 : buf1;
            hipLaunchKernelGGL(merge_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream, src,
                               dst, key_offsets, n_viewers, mt_off, r, o, c);
            e = hipGetLastError();
        }
        return e;
    }

    const int64_t cap = multi_cap(total);
    const Multi mt{mt_off, reinterpret_cast<int64_t *>(w + l.desc), cap,
                   reinterpret_cast<uint32_t *>(w + l.hist),
                   reinterpret_cast<uint64_t *>(w + l.status), counters,
                   reinterpret_cast<uint32_t *>(w + l.vclaim)};
    // Grids: one workgroup per viewer for the small-viewer kernel and per possible tile of the
    // multi-tile list for the others (the first two loop over any remainder; the first
    // kDirectPasses pass kernels take one tile per workgroup). Valid offsets give at most
    // total / kTile + B tiles (each multi-tile viewer adds at most one partial tile) and at most
    // cap < 2^22. Passes from kDirectPasses on, needed only for key spans above 27 bits, run on
    // a grid of kLoopGrid workgroups that claim tiles in a loop, so that their launches cost
    // little when they have nothing to do.
    const int64_t max_tiles = cap < total / kTile + n_viewers ? cap : total / kTile + n_viewers;
    const unsigned small_grid = (unsigned)(n_viewers < (1 << 16) ? n_viewers : (1 << 16));
    const unsigned hist_grid = (unsigned)(max_tiles < (1 << 20) ? max_tiles : (1 << 20));
    if (e == hipSuccess) {
        hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kThreads), 0, stream, key_offsets,
                           n_viewers, total, mt_off, slots, (int)n_slots, c, counters);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(small_kernel, dim3(small_grid), dim3(kThreads), 0, stream, keys_in,
                           key_offsets, n_viewers, mt, o, c);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(hist_kernel, dim3(hist_grid), dim3(kThreads), 0, stream, keys_in,
                           key_offsets, n_viewers, mt, o, c);
        e = hipGetLastError();
    }
    for (int p = 0; e == hipSuccess && p < c.max_passes; ++p) {
        const void *src = (p & 1) ? buf0 : buf1;     // written by pass p - 1
        void *dst = (p & 1) ? buf1 : buf0;
        if (p < kDirectPasses)
            hipLaunchKernelGGL(pass_kernel<false>, dim3((unsigned)max_tiles), dim3(kThreads), 0,
                               stream, keys_in, src, dst, key_offsets, n_viewers, mt, p, o, c);
        else
            hipLaunchKernelGGL(pass_kernel<true>, dim3(kLoopGrid), dim3(kThreads), 0, stream,
                               keys_in, src, dst, key_offsets, n_viewers, mt, p, o, c);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        const int64_t blocks = (total + kThreads - 1) / kThreads;
        hipLaunchKernelGGL(gather_kernel, dim3((unsigned)(blocks < (1 << 20) ? blocks : (1 << 20))),
                           dim3(kThreads), 0, stream, o);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace ccj
