// Alg. 1 Step 1 on the device (Connected Content Retriever §3.1): sort each viewer's affinity
// records by author id and move their feature rows with them.
//
// Each viewer's records (a CSR segment) are cut into tiles of kTile records. A record is sorted
// as an element that orders by (key, input position). That order is unique, so any correct sort
// is stable. Elements take one of two forms, chosen on the device for the whole call:
//   * packed, 8 bytes: ((key - kmin) << pbits) | (position within the viewer), when the span of
//     the call's keys leaves room for pbits position bits (pbits covers the largest viewer);
//     one 64-bit compare orders it, and it halves the bytes every pass moves;
//   * wide, 16 bytes: (key, flat input position), for any keys.
// Passes:
//   0. key range: the minimum and maximum key (per-workgroup slots, reduced by the plan), from
//      which every kernel derives the same form; plan: tile offsets per viewer (an exclusive
//      scan of ceil(K_v / kTile)).
//   1. block sort: a workgroup loads one tile; every thread sorts kEpt records in registers
//      with a bitonic network, then merge-path rounds in LDS double the sorted runs until the
//      tile's records are one run.
//   2. merge rounds: within each viewer, runs of kTile << r records are merged pairwise, one
//      output tile per workgroup. A viewer with n tiles takes part in ceil(log2 n) rounds. The
//      tile's two split points on the merge path are found by 64-ary searches, one wavefront
//      each (a few rounds of 64 probes instead of a ~20-step dependent binary search); the tile
//      is merged in LDS, kEpt outputs per thread.
//   3. A viewer's last pass (its block sort when it has one tile, else its last merge round)
//      writes the sorted keys and copies each record's feature row from the input, straight
//      from LDS; earlier passes write elements to two ping-pong arrays in a caller-provided
//      workspace.
// LDS rows are padded by one element every kEpt elements so that the per-thread blocked
// accesses (stride kEpt elements) spread over the banks. Other layouts (no padding, one pad per 16
// or 32 elements, XOR swizzles) timed the same within run-to-run noise: most of the LDS bank
// conflicts come from the data-dependent merge-path probes, which no static layout removes.
#include <stdint.h>

#include <mutex>

#include <hip/hip_runtime.h>

#include "join_internal.h"

namespace ccj {
namespace {

constexpr int kTile = 4096;                       // records per tile
constexpr int kThreads = 512;                     // threads per workgroup
constexpr int kEpt = kTile / kThreads;            // records per thread (8)
constexpr int kLdsElems = kTile + kTile / kEpt;   // padded LDS tile

typedef unsigned int chunk_t __attribute__((ext_vector_type(4)));

// Shared by every kernel of one call: the key range (written by range_kernel) and the number of
// position bits a packed element needs.
struct Codec {
    const int64_t *range;   // {min key, max key} in the workspace
    int32_t pbits;
};

struct Wide {
    struct T {
        int64_t key;
        int64_t f;    // flat input position
    };
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
};

struct Packed {
    typedef uint64_t T;
    int64_t kmin;
    int32_t pbits;
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
};

// Packed elements are usable when key - kmin < 2^(64 - pbits) - 1 for every key (the largest
// value stays free for padding). Every kernel evaluates this on the same range.
__device__ __forceinline__ bool use_packed(const Codec &c, int64_t &kmin) {
    kmin = c.range[0];
    const int64_t kmax = c.range[1];
    if (kmax < kmin)
        return true;                                    // no keys
    const uint64_t span = (uint64_t)kmax - (uint64_t)kmin;
    return span < (((uint64_t)1) << (64 - c.pbits)) - 1;
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
};

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
__global__ __launch_bounds__(kThreads) void plan_kernel(const int64_t *off, int32_t B,
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

// Records [base, base + n) go to the output unchanged (keys and rows, in input order).
__device__ __forceinline__ void copy_through(const int64_t *__restrict__ keys, int64_t base, int n,
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
            copy_through(keys, base, n, o);
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
        block_sort_body(Wide{}, lds, keys, off, B, tile_off, out, o);
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
        merge_body(Wide{}, lds, s_split, src, dst, off, B, tile_off, r, o);
}

constexpr int64_t round_up(int64_t x) { return (x + 255) & ~int64_t(255); }

constexpr int kRangeSlots = 1024;   // range_kernel workgroups at most

// Workspace layout: two ping-pong element arrays, the per-viewer tile offsets, the key range
// (256 bytes) and the range kernel's per-workgroup slots.
constexpr int64_t workspace_bytes(int64_t total, int64_t n_viewers) {
    return 2 * round_up(total * (int64_t)sizeof(Wide::T)) + round_up((n_viewers + 1) * 8) + 256 +
           round_up(2 * kRangeSlots * 8);
}

// Fixed device scratch of the allocation-free sort (cc_sort_affinity_noalloc): the workspace of
// the largest call it accepts. One copy per device, resolved once per device below; in host
// code `scratch` names a host-side stand-in, so only the resolved address is ever passed on.
constexpr int64_t kScratchBytes = workspace_bytes(kSortScratchRecords, kSortScratchViewers);
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

}  // namespace

int64_t sort_workspace_bytes(int64_t total, int32_t n_viewers) {
    // Counts the sort rejects (total >= 2^32) need no workspace; this also keeps the products
    // below far from overflow.
    if (total <= 0 || n_viewers <= 0 || total >= ((int64_t)1 << 32))
        return 0;
    return workspace_bytes(total, n_viewers);
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
                       int64_t *keys_out, void *rows_out, void *workspace, hipStream_t stream) {
    if (total <= 0 || n_viewers <= 0)
        return hipSuccess;
    uint8_t *w = static_cast<uint8_t *>(workspace);
    const int64_t buf_bytes = round_up(total * (int64_t)sizeof(Wide::T));
    void *buf0 = w;
    void *buf1 = w + buf_bytes;
    int64_t *tile_off = reinterpret_cast<int64_t *>(w + 2 * buf_bytes);
    int64_t *range =
        reinterpret_cast<int64_t *>(w + 2 * buf_bytes + round_up(((int64_t)n_viewers + 1) * 8));
    int64_t *slots = range + 32;                       // 256 bytes after range
    // Upper bound on tiles (every viewer adds at most one partial tile); larger counts are
    // covered by the kernels' grid-stride loops.
    int64_t grid = (total + kTile - 1) / kTile + n_viewers;
    if (grid > (1 << 20))
        grid = 1 << 20;
    const int64_t largest = max_keys > 0 ? (max_keys < total ? max_keys : total) : total;
    const int64_t per_viewer = (largest + kTile - 1) / kTile;
    int rounds = 0;
    while (((int64_t)1 << rounds) < per_viewer)
        ++rounds;
    // Position bits of a packed element: enough for the largest viewer.
    int32_t pbits = 1;
    while (((int64_t)1 << pbits) < largest)
        ++pbits;
    const Codec c{range, pbits};
    const SortOut o{largest, total, static_cast<const chunk_t *>(rows_in), row_bytes / 16,
                    keys_out, static_cast<chunk_t *>(rows_out)};
    int64_t n_slots = (total + kRangeThreads * kRangeUnroll - 1) / (kRangeThreads * kRangeUnroll);
    if (n_slots > kRangeSlots)
        n_slots = kRangeSlots;
    hipLaunchKernelGGL(range_kernel, dim3((unsigned)n_slots), dim3(kRangeThreads), 0, stream,
                       keys_in, total, slots);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) {
        hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kThreads), 0, stream, key_offsets,
                           n_viewers, total, tile_off, slots, (int)n_slots, range);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(block_sort_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream,
                           keys_in, key_offsets, n_viewers, tile_off, buf0, o, c);
        e = hipGetLastError();
    }
    for (int r = 0; e == hipSuccess && r < rounds; ++r) {
        const void *src = (r & 1) ? buf1 : buf0;
        void *dst = (r & 1) ? buf0 : buf1;
        hipLaunchKernelGGL(merge_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream, src, dst,
                           key_offsets, n_viewers, tile_off, r, o, c);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace ccj
