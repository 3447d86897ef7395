// Edge-feature join kernels for gfx950 (CDNA4).
//
// Operation: Connected Content Retriever §3.1, Eq. 1 with the search of Alg. 1 Steps 2-4,
// fused with the gather of the candidate's document row (§6.3). The path is a memory-bound
// search-and-copy: no matrix cores, no arithmetic on the row payloads.
//
// Work decomposition
//   * The flattened candidate array [0, total_cand) is cut into n_wg contiguous ranges of
//     per_wg candidates. Hardware dispatches workgroup b to XCD b % 8, so the range index is
//     (b % 8) * (n_wg / 8) + b / 8: each XCD walks one contiguous eighth of the candidates,
//     which keeps a viewer's keys and edge rows in a single XCD's L2.
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
//            read those (at most S) keys from global memory (L2) in one step and count.
//   hit    : some key equal to x in the inspected window; because keys ascend, the lower
//            bound is then the leftmost equal key.
#include "join_internal.h"

namespace ccj {
namespace {

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
    const int64_t lo = (g - 1) * S + 1;
    const int64_t hi = min(g * (int64_t)S, K);
    const int64_t *w = gk + lo;
    int64_t len = hi - lo;
    // Wide strides (only when K exceeds 16x the LDS table): narrow in global memory first.
    while (len > kWindow) {
        const int64_t half = len >> 1;
        w = (w[half] < x) ? w + half : w;
        len -= half;
    }
    // The lower bound lies in [w, w + len]; inspect w[0..len] (w[len] may be past the end).
    const int64_t avail = (gk + K) - w;
    int64_t cnt = 0;
    bool eq = false;
#pragma unroll
    for (int t = 0; t <= kWindow; ++t) {
        if (t <= len && t < avail) {
            const int64_t k = w[t];
            cnt += (t < len && k < x) ? 1 : 0;
            eq |= (k == x);
        }
    }
    return eq ? (w - gk) + cnt : -1;
}

// Fence stride for one segment: the smallest power of two whose fence count fits the LDS
// table and is not much larger than the number of candidates that will use it.
__device__ __forceinline__ int choose_stride(int64_t K, int64_t seg_len, int32_t cap,
                                             int32_t forced) {
    int64_t budget = forced > 0 ? cap : min<int64_t>(cap, max<int64_t>(512, 4 * seg_len));
    int S = forced > 0 ? forced : 1;
    while ((K + S - 1) / S > budget)
        S <<= 1;
    return S;
}

__device__ __forceinline__ int64_t range_index(int b, int n) {
    const int per_xcd = n >> 3;
    return (int64_t)(b & 7) * per_xcd + (b >> 3);
}

// Copy one sub-tile's output rows. DOC_CH / EDGE_CH are row widths in 16-byte chunks
// (0 = read them from the arguments).
template <int DOC_CH, int EDGE_CH, int NL>
__device__ __forceinline__ void copy_rows(const JoinArgs &a, const int64_t *s_src,
                                          const int64_t (*s_row)[kBlock], int64_t t0, int n) {
    const int tid = threadIdx.x;
    if constexpr (DOC_CH > 0) {
        constexpr int CH = DOC_CH + NL * EDGE_CH;
        uint4 v[CH];
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int e = i * kBlock + tid;
            const int row = e / CH;
            const int k = e - row * CH;
            v[i] = make_uint4(0u, 0u, 0u, 0u);
            if (row < n) {
                const uint4 *src = nullptr;
                if (k < DOC_CH) {
                    const int64_t c = s_src[row];
                    if (c >= 0)
                        src = reinterpret_cast<const uint4 *>(a.doc + c * (DOC_CH * 16)) + k;
                } else {
                    const int kk = k - DOC_CH;
                    const int l = kk / EDGE_CH;
                    const int q = kk - l * EDGE_CH;
                    const int64_t r = s_row[l][row];
                    if (r >= 0)
                        src = reinterpret_cast<const uint4 *>(a.edge + r * (EDGE_CH * 16)) + q;
                    else if (a.def_row)
                        src = reinterpret_cast<const uint4 *>(a.def_row) + q;
                }
                if (src)
                    v[i] = *src;
            }
        }
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int e = i * kBlock + tid;
            const int row = e / CH;
            const int k = e - row * CH;
            if (row < n)
                reinterpret_cast<uint4 *>(a.out + (t0 + row) * a.out_stride)[k] = v[i];
        }
    } else {
        const int dch = a.doc_bytes >> 4;
        const int ech = a.edge_bytes >> 4;
        const int ch = dch + NL * ech;
        const int total = n * ch;
        constexpr int U = 4;
        for (int base = 0; base < total; base += U * kBlock) {
            uint4 v[U];
            int rows[U], ks[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = base + u * kBlock + tid;
                rows[u] = e / ch;
                ks[u] = e - rows[u] * ch;
                v[u] = make_uint4(0u, 0u, 0u, 0u);
                if (e < total) {
                    const int row = rows[u], k = ks[u];
                    const uint4 *src = nullptr;
                    if (k < dch) {
                        const int64_t c = s_src[row];
                        if (c >= 0)
                            src = reinterpret_cast<const uint4 *>(a.doc + c * a.doc_bytes) + k;
                    } else {
                        const int kk = k - dch;
                        const int l = kk / ech;
                        const int q = kk - l * ech;
                        const int64_t r = s_row[l][row];
                        if (r >= 0)
                            src = reinterpret_cast<const uint4 *>(a.edge + r * a.edge_bytes) + q;
                        else if (a.def_row)
                            src = reinterpret_cast<const uint4 *>(a.def_row) + q;
                    }
                    if (src)
                        v[u] = *src;
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = base + u * kBlock + tid;
                if (e < total)
                    reinterpret_cast<uint4 *>(a.out + (t0 + rows[u]) * a.out_stride)[ks[u]] = v[u];
            }
        }
    }
}

template <int DOC_CH, int EDGE_CH, int NL>
__global__ __launch_bounds__(kBlock) void join_kernel(JoinArgs a) {
    extern __shared__ int64_t s_tab[];            // fence table, a.lds_keys entries
    __shared__ int64_t s_src[kBlock];             // doc position of each sub-tile row, or -1
    __shared__ int64_t s_row[NL][kBlock];         // global edge row per lookup, or -1
    __shared__ unsigned int s_invalid;

    const int tid = threadIdx.x;
    int64_t begin = range_index(blockIdx.x, gridDim.x) * a.per_wg;
    const int64_t end = min(begin + a.per_wg, a.total_cand);
    if (begin >= end)
        return;
    if (tid == 0)
        s_invalid = 0;

    const bool batched = a.cand_offsets != nullptr;
    const int32_t B = batched ? a.n_viewers : 1;
    // First viewer whose candidate range ends after `begin`.
    int32_t v = 0;
    if (batched) {
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

    for (; v < B && begin < end; ++v) {
        int64_t vb = 0, ve = a.total_cand, kb = 0, ke = a.total_keys;
        if (batched) {
            vb = clamp64(a.cand_offsets[v], a.total_cand);
            ve = clamp64(a.cand_offsets[v + 1], a.total_cand);
            kb = clamp64(a.key_offsets[v], a.total_keys);
            ke = max(kb, clamp64(a.key_offsets[v + 1], a.total_keys));
        }
        const int64_t s0 = max(begin, vb);
        const int64_t s1 = min(end, ve);
        if (s1 <= s0)
            continue;
        begin = s1;

        const int64_t K = ke - kb;
        const int64_t *gk = a.keys + kb;
        const int S = choose_stride(K, s1 - s0, a.lds_keys, a.fence_stride);
        const int64_t M = (K + S - 1) / S;
        __syncthreads();                          // earlier readers of s_tab are done
        for (int64_t i = tid; i < M; i += kBlock)
            s_tab[i] = gk[i * S];
        __syncthreads();

        for (int64_t t0 = s0; t0 < s1; t0 += kBlock) {
            const int n = (int)min<int64_t>(kBlock, s1 - t0);
            if (tid < n) {
                const int64_t j = t0 + tid;
                const int64_t c = a.cand_idx[j];
                const bool valid = c >= 0 && c < a.n_docs;
                s_src[tid] = valid ? c : -1;
                if (!valid)
                    atomicAdd(&s_invalid, 1u);
#pragma unroll
                for (int l = 0; l < NL; ++l) {
                    int64_t r = -1;
                    if (valid) {
                        const int64_t x = (l == 0) ? a.author[c] : a.extra[j];
                        r = find_key(x, s_tab, M, S, gk, K);
                    }
                    s_row[l][tid] = r >= 0 ? kb + r : -1;
                    a.hit[j * NL + l] = (int8_t)(r >= 0 ? 1 : 0);
                }
            }
            __syncthreads();
            copy_rows<DOC_CH, EDGE_CH, NL>(a, s_src, s_row, t0, n);
            __syncthreads();
        }
    }
    if (tid == 0 && s_invalid)
        atomicAdd(a.invalid_counter, (unsigned long long)s_invalid);
}

template <int D, int E, int L>
hipError_t launch_one(const JoinArgs &a, hipStream_t stream) {
    const size_t lds = (size_t)max(1, a.lds_keys) * sizeof(int64_t);
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&join_kernel<D, E, L>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess)
            return e;
    }
    hipLaunchKernelGGL((join_kernel<D, E, L>), dim3(a.n_wg), dim3(kBlock), lds, stream, a);
    return hipGetLastError();
}

template <int L>
hipError_t dispatch_widths(const JoinArgs &a, hipStream_t stream) {
    const int d = a.doc_bytes >> 4, e = a.edge_bytes >> 4;
    if (d == 4 && e == 2) return launch_one<4, 2, L>(a, stream);
    if (d == 8 && e == 4) return launch_one<8, 4, L>(a, stream);
    if (d == 8 && e == 8) return launch_one<8, 8, L>(a, stream);
    return launch_one<0, 0, L>(a, stream);
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

hipError_t launch_join(const JoinArgs &a, int n_lookups, hipStream_t stream) {
    return n_lookups == 2 ? dispatch_widths<2>(a, stream) : dispatch_widths<1>(a, stream);
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
