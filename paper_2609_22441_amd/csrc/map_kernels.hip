// Document-id map on the device: H(id) -> store position (Connected Content Retriever §6.3.1,
// Eq. 6) and the ingestion batch that maintains it (§6.2, bootstrap protocol).
//
// The paper keeps H as a CPU hash map because a GPU hash map would need rebuilds under tens
// of thousands of upserts per second. Here the map is an open-addressing table in HBM sized
// for a load factor of at most 1/2 of the store's capacity, so an upsert never rebuilds it:
// new ids are placed with a compare-and-swap and stored ids are found in place.
//
// Layout: groups of kGroup 16-byte entries (64 bytes); an id probes groups h, h+1, ... from
// its home group h = mix(id) mod n_groups and takes the first free entry. Entries are only
// ever freed by the rollback of a batch that did not fit, and those entries were free before
// the batch, so the occupied entries of a group always form a prefix and an id that is absent
// is known to be absent at the first group with a free entry. Probing stops after
// kMaxProbeGroups groups; an id that cannot be placed within that distance fails its batch.
//
// Ingestion batch of n records (§6.2: identify new vs. stored ids, prefix-sum positions for the
// new ones, scatter rows, update the map only after the rows are written):
//   claim:   every record finds or claims its id's entry, which then holds the first record
//            index (pos = -(3 + i), only while the entry is pending) and the last record index
//            (aux): the record whose swap put a new id into the entry sets both with one
//            write-through store, its repeats wait for that store and fold in with atomic
//            maxima; an exclusive scan over "record i is the first occurrence of a new id"
//            (one pass, tiles chained by decoupled look-back) gives each new id its rank, in
//            batch order.
//   apply:   the last occurrence of every id copies its row and author id to the stored
//            position or to n_old + rank; then the first occurrence commits pos and every
//            record clears aux.
//   rollback (batch does not fit): pending entries are freed again, aux is cleared.
// Whether the batch fits (every id placed, n_old + n_new <= capacity) is decided on the device
// from the claim's counts: apply and rollback are both enqueued and each does nothing unless
// it is the one that applies, so a batch needs a single synchronisation at its end.
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "join_internal.h"

namespace ccj {
namespace {

constexpr int kThreads = 256;
// Records per thread in a scan tile: large batches take big tiles (fewer tiles to chain), small
// ones small tiles (more workgroups, shorter per-tile chains).
constexpr int kScanPerLarge = 32;
constexpr int kScanPerSmall = 4;
constexpr int64_t kScanLargeFrom = 1 << 22;        // records
__host__ __device__ inline int scan_per(int64_t n) {
    return n >= kScanLargeFrom ? kScanPerLarge : kScanPerSmall;
}
constexpr uint64_t kMaxProbeGroups = 64;
// counts[]: new ids, rejected records, unplaced ids, author ids wider than 32 bits, the scan's
// tile counter, waits (of the claim or the scan) that reached their bound of max_polls polls.
constexpr int kCounts = kUpsertCounts;
static_assert(kCounts * 8 <= 256, "the counts live in the workspace's last 256 bytes");

typedef unsigned int chunk_t __attribute__((ext_vector_type(4)));

// SplitMix64 output function (Steele, Lea and Flood 2014; Vigna's constants): a bijective
// 64-bit mixer, so that ids that differ in any bit spread over the groups.
__device__ __forceinline__ uint64_t mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

__device__ __forceinline__ int64_t load_key(const MapEntry *e) {
    return __hip_atomic_load(&e->key, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int64_t grid_stride() { return (int64_t)gridDim.x * blockDim.x; }

__device__ __forceinline__ int64_t global_id() {
    return (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
}

// Workspace: slot int64[n] | rank int32[n] | posv int32[n] | last uint8[n] | dup uint8[n] |
// status uint64[blocks] | counts int64[kCounts].
//   slot   map entry of record i (-1: reserved id or not placed)
//   posv   the entry's position field once every record has claimed: a stored position >= 0,
//          or -(3 + first record) for an id new in this batch, or kNoPos when slot < 0
//   last   1 when record i is the last record with its id (it carries the row to store)
//   dup    1 when another record of the batch has record i's id. The claim writes posv and
//          last as they are for an id without repeats (and kNoPos, 0 for a record without an
//          entry); the scan reads the map entry only for the records marked here.
//   status the scan's look-back word of each tile of kThreads * scan_per(n) records (cleared
//          per batch; sized for the small tiles)
struct Ws {
    int64_t *slot;
    int32_t *rank;
    int32_t *posv;
    uint8_t *last;
    uint8_t *dup;
    uint64_t *status;
    int64_t *counts;     // kCounts entries (see kCounts)
    int64_t blocks;
};

__host__ __device__ int64_t round_up(int64_t x) { return (x + 255) & ~int64_t(255); }

Ws carve(void *workspace, int64_t n) {
    uint8_t *w = static_cast<uint8_t *>(workspace);
    Ws s;
    s.blocks = (n + kThreads * scan_per(n) - 1) / (kThreads * scan_per(n));
    s.slot = reinterpret_cast<int64_t *>(w);
    w += round_up(n * 8);
    s.rank = reinterpret_cast<int32_t *>(w);
    w += round_up(n * 4);
    s.posv = reinterpret_cast<int32_t *>(w);
    w += round_up(n * 4);
    s.last = w;
    w += round_up(n);
    s.dup = w;
    w += round_up(n);
    s.status = reinterpret_cast<uint64_t *>(w);
    w += round_up((n + kThreads * kScanPerSmall - 1) / (kThreads * kScanPerSmall) * 8);
    s.counts = reinterpret_cast<int64_t *>(w);
    return s;
}

__global__ void map_init_kernel(MapEntry *map, int64_t n_entries) {
    for (int64_t i = global_id(); i < n_entries; i += grid_stride())
        map[i] = MapEntry{kEmptyKey, kNoPos, -1};
}

// One query per quad of lanes: each lane reads one entry of the probed group (a quad reads the
// group's 64 contiguous bytes) and the quad votes. A quad takes kResolvePer queries at a time and
// issues their first-group reads together, so each wavefront keeps several HBM round trips in
// flight; the rare query whose first group is full and does not hold its id probes on alone.
constexpr int kResolvePer = 4;

__device__ __forceinline__ bool quad_vote(const MapEntry &e, int64_t key, int quad0,
                                          int64_t &result) {
    const unsigned hit = (unsigned)(__ballot(e.key == key) >> quad0) & 0xF;
    const unsigned emp = (unsigned)(__ballot(e.key == kEmptyKey) >> quad0) & 0xF;
    if (hit) {
        const int32_t p = __shfl(e.pos, quad0 + __builtin_ctz(hit));
        result = p >= 0 ? p : -1;
        return true;
    }
    return emp != 0;                              // a free entry ends the probe: absent
}

__global__ __launch_bounds__(kThreads) void resolve_kernel(const MapEntry *__restrict__ map,
                                                           uint64_t mask,
                                                           const int64_t *__restrict__ ids,
                                                           int64_t n, int64_t *__restrict__ pos) {
    const int lane = threadIdx.x & 63;
    const int sub = lane & (kGroup - 1);
    const int quad0 = lane & ~(kGroup - 1);
    const int64_t stride = grid_stride() / kGroup;
    for (int64_t q0 = global_id() / kGroup; q0 < n; q0 += kResolvePer * stride) {
        int64_t key[kResolvePer];
        uint64_t g[kResolvePer];
        MapEntry e[kResolvePer];
#pragma unroll
        for (int r = 0; r < kResolvePer; ++r) {
            const int64_t q = q0 + r * stride;
            key[r] = q < n ? ids[q] : kEmptyKey;
            g[r] = mix((uint64_t)key[r]) & mask;
        }
#pragma unroll
        for (int r = 0; r < kResolvePer; ++r)
            e[r] = map[g[r] * kGroup + sub];      // in bounds for every key, used or not
#pragma unroll
        for (int r = 0; r < kResolvePer; ++r) {
            const int64_t q = q0 + r * stride;
            if (q >= n)
                break;                            // uniform per quad
            int64_t result = -1;
            if (key[r] != kEmptyKey && !quad_vote(e[r], key[r], quad0, result)) {
                uint64_t gg = g[r];
                for (uint64_t probe = 1; probe < kMaxProbeGroups && probe <= mask; ++probe) {
                    gg = (gg + 1) & mask;
                    if (quad_vote(map[gg * kGroup + sub], key[r], quad0, result))
                        break;
                }
            }
            if (sub == 0)
                pos[q] = result;
        }
    }
}

// Clears the batch's counts, its repeat marks (round_up(n) bytes, 16 at a time) and the scan's
// look-back words.
__global__ void counts_init_kernel(Ws w, int64_t n) {
    if (blockIdx.x == 0 && threadIdx.x < kCounts)
        w.counts[threadIdx.x] = 0;
    const int64_t chunks = round_up(n) / 16;
    for (int64_t c = global_id(); c < chunks; c += grid_stride())
        reinterpret_cast<chunk_t *>(w.dup)[c] = chunk_t{0u, 0u, 0u, 0u};
    for (int64_t b = global_id(); b < w.blocks; b += grid_stride())
        w.status[b] = 0;
}

// One record per quad of lanes: each lane reads one entry of the probed group (the quad reads
// the group's 64 contiguous bytes in one instruction) and the quad votes. A group holding the id
// ends the probe; otherwise the quad claims the group's first free entry with one
// compare-and-swap (entries before it are occupied, so the occupied entries stay a prefix of
// the probe order). A failed swap that returns another id means that entry was just taken:
// the group is read again, at most kGroup times in all. A group with no free entry sends the
// probe on to the next one. Then one lane records the first and last record in the entry and
// writes the record's workspace fields as they are for an id without repeats (see Ws). The
// entry's key and its position word are separate 8-byte words, so a new id costs one swap (the
// key) and one store; a second swap for the position word would be a second round trip past L2.
__global__ __launch_bounds__(kThreads) void claim_kernel(MapEntry *map, uint64_t mask,
                                                         const int64_t *__restrict__ ids,
                                                         int64_t n, Ws w, int32_t max_polls) {
    const int lane = threadIdx.x & 63;
    const int sub = lane & (kGroup - 1);
    const int quad0 = lane & ~(kGroup - 1);
    const int64_t stride = grid_stride() / kGroup;
    for (int64_t i = global_id() / kGroup; i < n; i += stride) {      // uniform per quad
        const int64_t key = ids[i];
        if (key == kEmptyKey) {
            if (sub == 0) {
                atomicAdd(reinterpret_cast<unsigned long long *>(&w.counts[1]), 1ULL);
                w.slot[i] = -1;
                w.posv[i] = kNoPos;
                w.last[i] = 0;
            }
            continue;
        }
        uint64_t g = mix((uint64_t)key) & mask;
        int64_t found = -1;
        bool created = false;             // this record's swap put the id into the entry
        bool stored = false;              // the id was stored by an earlier batch
        int32_t stored_pos = kNoPos;      // its position then
        uint64_t probe = 0;
        int retries = 0;
        while (probe < kMaxProbeGroups && probe <= mask) {
            MapEntry *grp = map + g * kGroup;
            const int64_t k = load_key(grp + sub);
            const unsigned hit = (unsigned)(__ballot(k == key) >> quad0) & 0xF;
            if (hit) {
                found = (int64_t)(g * kGroup) + __builtin_ctz(hit);
                // A position >= 0 was committed by an earlier batch and does not change during
                // this one (only entries claimed in this batch carry pending values).
                stored_pos = __shfl(grp[sub].pos, quad0 + __builtin_ctz(hit));
                stored = stored_pos >= 0;
                break;
            }
            const unsigned emp = (unsigned)(__ballot(k == kEmptyKey) >> quad0) & 0xF;
            if (!emp || retries == kGroup) {
                g = (g + 1) & mask;
                ++probe;
                retries = 0;
                continue;
            }
            const int e = __builtin_ctz(emp);
            unsigned long long got = 0;
            if (sub == e)
                got = atomicCAS(reinterpret_cast<unsigned long long *>(&grp[e].key),
                                (unsigned long long)kEmptyKey, (unsigned long long)key);
            got = __shfl(got, quad0 + e);
            if ((int64_t)got == kEmptyKey || (int64_t)got == key) {
                found = (int64_t)(g * kGroup) + e;         // claimed now, or by the same id
                created = (int64_t)got == kEmptyKey;
                break;
            }
            ++retries;                                     // another id took entry e
        }
        // A record that put a new id into the entry publishes its first and last record with
        // one write-through store: no other record of the batch writes that word before it
        // (they wait for it below). This runs as a region of its own, ahead of the waits, so
        // that a creator and a repeat of its id in one wavefront (whose divergent branches run
        // one after the other) never leave the wait spinning before the store.
        if (sub == 0 && found >= 0 && created) {
            const unsigned long long mine =
                (unsigned long long)(uint32_t)(-(3 + (int32_t)i)) |
                ((unsigned long long)(uint32_t)(int32_t)i << 32);
            static_assert(offsetof(MapEntry, aux) == offsetof(MapEntry, pos) + 4,
                          "pos and aux share one 8-byte word");
            w.slot[i] = found;
            w.posv[i] = -(3 + (int32_t)i);
            w.last[i] = 1;
            __hip_atomic_store(reinterpret_cast<unsigned long long *>(&map[found].pos), mine,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (sub == 0 && !(found >= 0 && created)) {
            w.slot[i] = found;
            if (found < 0) {
                atomicAdd(reinterpret_cast<unsigned long long *>(&w.counts[2]), 1ULL);
                w.posv[i] = kNoPos;
                w.last[i] = 0;
            } else if (stored) {
                // Atomics on device memory are performed past the per-XCD L2 caches, so each
                // costs a memory round trip: a stored entry's position needs none. The old
                // last record comes back: -1 while this is the id's only record so far,
                // otherwise a record of the same id, which this one marks with itself.
                w.posv[i] = stored_pos;
                w.last[i] = 1;
                const int32_t prev = atomicMax(&map[found].aux, (int32_t)i);
                if (prev >= 0) {
                    w.dup[i] = 1;
                    w.dup[prev] = 1;
                }
            } else {
                // A repeat of an id that another record of this batch put into the entry: wait
                // until that record's store is visible (its values replace the idle ones; the
                // creator stores right after its swap), then fold this record in with two
                // maxima. The first repeat to read sees the creator's values, so every record
                // of a repeated id ends up marked. A wait that reaches its bound is counted in
                // counts[5]: the first and last record may then be wrong, and the batch is
                // refused and rolled back (pending entries are freed whatever they hold).
                const unsigned long long idle =
                    (unsigned long long)(uint32_t)kNoPos | ((unsigned long long)(uint32_t)-1 << 32);
                unsigned long long old = idle;
                for (int polls = 0; polls < max_polls; ++polls) {
                    old = __hip_atomic_load(reinterpret_cast<unsigned long long *>(&map[found].pos),
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (old != idle)
                        break;
                    __builtin_amdgcn_s_sleep(1);
                }
                if (old == idle)
                    atomicAdd(reinterpret_cast<unsigned long long *>(&w.counts[5]), 1ULL);
                w.posv[i] = -(3 + (int32_t)i);
                w.last[i] = 1;
                atomicMax(&map[found].pos, -(3 + (int32_t)i));
                atomicMax(&map[found].aux, (int32_t)i);
                const int32_t p = (int32_t)(uint32_t)old;
                const int32_t q = (int32_t)(uint32_t)(old >> 32);
                w.dup[i] = 1;
                if (p <= -3 && -(int64_t)p - 3 < n)
                    w.dup[-(int64_t)p - 3] = 1;
                if (q >= 0 && q < n)
                    w.dup[q] = 1;
            }
        }
    }
}

// Record i is the first occurrence of an id that is new in this batch (posv already read).
__device__ __forceinline__ int32_t first_new(const Ws &w, int64_t i) {
    return w.posv[i] == -(3 + (int32_t)i) ? 1 : 0;
}

// Look-back word of one scan tile: flag in the top two bits (0 = not yet published, kAgg = the
// tile's own count of new ids, kInc = the count over this and every earlier tile), the count
// below them.
constexpr uint64_t kAgg = (uint64_t)1 << 62;
constexpr uint64_t kInc = (uint64_t)2 << 62;
constexpr uint64_t kCountMask = kAgg - 1;

__device__ __forceinline__ void put_status(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t get_status(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int64_t wave_sum(int64_t x) {
    for (int off = 32; off > 0; off >>= 1)
        x += __shfl_xor(x, off);
    return x;
}

// New ids in tiles 0 .. k (k >= 0), by one whole wavefront: lane l reads the word of tile
// k - l, so each round trip inspects 64 tiles; the words up to the nearest inclusive one are
// added, else all 64 and the window moves down. Tiles below 0 read as inclusive zeros (tile 0
// itself always publishes an inclusive word). Each tile waits only for tiles claimed before
// it, by workgroups that publish their own count before they look back, so a wait lasts about
// one tile's loads. A word still unpublished after max_polls polls ends the walk and is counted
// in counts[5]: the batch is then refused and rolled back. Every lane returns the sum.
__device__ int64_t look_back(const Ws &w, int64_t k, int32_t max_polls) {
    const int lane = threadIdx.x & 63;
    int64_t sum = 0;
    int polls = 0;
    while (true) {
        const int64_t t = k - lane;
        uint64_t v = t >= 0 ? get_status(w.status + t) : kInc;
        while (__ballot((v & ~kCountMask) == 0) != 0 && polls < max_polls) {
            ++polls;
            __builtin_amdgcn_s_sleep(1);
            if ((v & ~kCountMask) == 0)
                v = get_status(w.status + t);
        }
        if (__ballot((v & ~kCountMask) == 0) != 0) {
            if (lane == 0)
                atomicAdd(reinterpret_cast<unsigned long long *>(&w.counts[5]), 1ULL);
            return sum;
        }
        const uint64_t inc = __ballot((v & ~kCountMask) == kInc);
        if (inc != 0) {
            const int m = __builtin_ctzll(inc);      // nearest inclusive word
            return sum + wave_sum(lane <= m ? (int64_t)(v & kCountMask) : 0);
        }
        sum += wave_sum((int64_t)(v & kCountMask));
        k -= 64;
    }
}

// The scan, in one pass with decoupled look-back. A workgroup claims the next tile of
// kThreads * PER records from counts[4] (so every tile it waits for belongs to a workgroup that is
// already running), reads each record's entry position (from the workspace; from the map for a
// record marked as a repeat, which also gives its last mark: the one read of the map after the
// claim, so that later passes read the workspace in order), counts the first occurrences of
// new ids with one ballot per wavefront and round, publishes the tile's count, looks back for
// the count before the tile, and writes rank[i] = number of first occurrences of new ids
// before record i. Records are read in rounds of kThreads consecutive ones (coalesced); the
// rank order inside a tile is round, then wavefront, then lane, which is record order.
template <int PER>
__global__ __launch_bounds__(kThreads) void scan_kernel(const MapEntry *map, int64_t n, Ws w,
                                                        int32_t max_polls) {
    __shared__ int64_t s_tile, s_before;
    __shared__ int32_t s_cnt[PER][kThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0)
        s_tile = (int64_t)atomicAdd(reinterpret_cast<unsigned long long *>(&w.counts[4]), 1ULL);
    __syncthreads();
    const int64_t tile = s_tile;
    const int64_t base = tile * (kThreads * PER);
    // The position fields and marks of all rounds are loaded at once, from clamped indices (a
    // load under a branch would be waited for before the next round's loads are issued). A
    // record without repeats needs nothing else: the claim wrote its position field and last
    // mark. A repeat reads its entry index and the entry (whose pos gives the id's first record
    // and aux its last), in a branch that wavefronts without repeats skip.
    static_assert(PER <= 32, "one bit per round in a 32-bit mask");
    int32_t pv[PER];
    uint32_t dup = 0;                             // bit k: round k's record is a repeat
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int64_t i = min(base + k * kThreads + tid, n - 1);
        pv[k] = w.posv[i];
        dup |= (w.dup[i] && base + k * kThreads + tid < n ? 1u : 0u) << k;
    }
    uint32_t dup_first = 0;                       // bit k: ... and the first of its id
    if (__ballot(dup != 0) != 0) {
        // kDupRounds rounds at a time: their entry indices, then their entries, each group of
        // loads issued together (from clamped indices: the tile's first record and entry 0
        // for records that are not repeats).
        constexpr int kDupRounds = PER < 8 ? PER : 8;
        static_assert(PER % kDupRounds == 0, "whole groups of rounds");
        const int64_t i0 = min(base, n - 1);
#pragma unroll 1
        for (int c = 0; c < PER; c += kDupRounds) {
            int64_t sl[kDupRounds];
#pragma unroll
            for (int u = 0; u < kDupRounds; ++u) {
                const bool d = (dup >> (c + u)) & 1u;
                sl[u] = w.slot[d ? base + (c + u) * kThreads + tid : i0];
            }
            int32_t ep[kDupRounds], ea[kDupRounds];
#pragma unroll
            for (int u = 0; u < kDupRounds; ++u) {
                const bool d = (dup >> (c + u)) & 1u;
                const MapEntry &m = map[d && sl[u] >= 0 ? sl[u] : 0];
                ep[u] = m.pos;
                ea[u] = m.aux;
            }
#pragma unroll
            for (int u = 0; u < kDupRounds; ++u) {
                const int64_t i = base + (c + u) * kThreads + tid;
                if ((dup >> (c + u)) & 1u) {            // a repeat always has an entry
                    w.posv[i] = ep[u];
                    w.last[i] = ea[u] == (int32_t)i ? 1 : 0;
                    dup_first |= (ep[u] == -(3 + (int32_t)i) ? 1u : 0u) << (c + u);
                }
            }
        }
    }
    uint64_t bal[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int64_t i = base + k * kThreads + tid;
        const bool first = i < n && (((dup >> k) & 1u) ? ((dup_first >> k) & 1u) != 0
                                                        : pv[k] == -(3 + (int32_t)i));
        bal[k] = __ballot(first);
        if (lane == 0)
            s_cnt[k][wave] = __popcll(bal[k]);
    }
    __syncthreads();
    if (wave == 0) {
        int64_t tot = 0;
        for (int k = 0; k < PER; ++k)
            for (int v = 0; v < kThreads / 64; ++v)
                tot += s_cnt[k][v];
        int64_t before = 0;
        if (tile == 0) {
            if (lane == 0)
                put_status(w.status, kInc | (uint64_t)tot);
        } else {
            if (lane == 0)
                put_status(w.status + tile, kAgg | (uint64_t)tot);
            before = look_back(w, tile - 1, max_polls);
            if (lane == 0)
                put_status(w.status + tile, kInc | (uint64_t)(before + tot));
        }
        if (lane == 0) {
            if (tile == w.blocks - 1)
                w.counts[0] = before + tot;        // new ids in the batch
            s_before = before;
        }
    }
    __syncthreads();
    int64_t run = s_before;
    const uint64_t below = (lane == 0) ? 0ULL : (~0ULL >> (64 - lane));
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        int32_t waves_before = 0, round = 0;
        for (int v = 0; v < kThreads / 64; ++v) {
            const int32_t c = s_cnt[k][v];
            waves_before += v < wave ? c : 0;
            round += c;
        }
        const int64_t i = base + k * kThreads + tid;
        if (i < n)
            w.rank[i] = (int32_t)(run + waves_before + __popcll(bal[k] & below));
        run += round;
    }
}

// The batch fits: every id was placed, the new ids fit in the remaining capacity and no wait of
// the scan reached its bound.
__device__ __forceinline__ bool batch_fits(const Ws &w, int64_t n_old, int64_t capacity) {
    return w.counts[2] == 0 && w.counts[5] == 0 && n_old + w.counts[0] <= capacity;
}

__global__ void rollback_kernel(MapEntry *map, int64_t n, Ws w, int64_t n_old, int64_t capacity) {
    if (batch_fits(w, n_old, capacity))
        return;
    for (int64_t i = global_id(); i < n; i += grid_stride()) {
        const int64_t s = w.slot[i];
        if (s < 0)
            continue;
        if (map[s].pos < 0) {                     // pending: claimed by this batch
            map[s].key = kEmptyKey;
            map[s].pos = kNoPos;
        }
        map[s].aux = -1;
    }
}

// The last occurrence of each id writes its row and author id, at the stored position or at
// n_old + the rank of the id's first record. A thread takes kScatterPer 16-byte chunks of its
// grid-stride sequence at a time and issues their loads in three rounds (last marks; position
// fields, row chunks and author ids; ranks of new ids), so that each round trip serves
// kScatterPer chunks; a chunk's record and column advance by the stride without a division.
constexpr int kScatterPer = 4;

__global__ __launch_bounds__(kThreads) void scatter_kernel(int64_t n, Ws w,
                                                           int64_t n_old, int64_t capacity,
                                                           const int64_t *__restrict__ author_in,
                                                           const chunk_t *__restrict__ rows_in,
                                                           int32_t chunks,
                                                           int64_t *__restrict__ author,
                                                           int32_t *__restrict__ author32,
                                                           chunk_t *__restrict__ rows) {
    if (!batch_fits(w, n_old, capacity))
        return;
    constexpr int U = kScatterPer;
    const int64_t total = n * chunks;
    const int64_t stride = grid_stride();
    const int64_t di = stride / chunks;
    const int32_t dq = (int32_t)(stride - di * chunks);
    int64_t i = global_id() / chunks;
    int32_t q = (int32_t)(global_id() - i * chunks);
    for (int64_t g = global_id(); g < total; g += U * stride) {
        int64_t rec[U];
        int32_t col[U];
        bool in[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            rec[u] = i;
            col[u] = q;
            in[u] = g + u * stride < total;
            i += di;
            q += dq;
            if (q >= chunks) {
                q -= chunks;
                ++i;
            }
        }
        bool carry[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            carry[u] = in[u] && w.last[rec[u]];   // a later record carries this id's row
        int32_t pv[U];
        chunk_t c[U];
        int64_t x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            pv[u] = 0;
            x[u] = 0;
            if (carry[u]) {
                pv[u] = w.posv[rec[u]];
                c[u] = rows_in[rec[u] * chunks + col[u]];
                if (col[u] == 0)
                    x[u] = author_in[rec[u]];
            }
        }
        int64_t target[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            target[u] = !carry[u] || pv[u] >= 0 ? (int64_t)pv[u]
                                                : n_old + w.rank[-(int64_t)pv[u] - 3];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (!carry[u])
                continue;
            rows[target[u] * chunks + col[u]] = c[u];
            if (col[u] == 0) {
                author[target[u]] = x[u];
                author32[target[u]] = (int32_t)x[u];
                if (x[u] < INT32_MIN || x[u] > INT32_MAX)
                    atomicAdd(reinterpret_cast<unsigned long long *>(&w.counts[3]), 1ULL);
            }
        }
    }
}

// The map changes only now, after the rows are written: the first record of a new id stores
// its position, the last record of every id clears the entry's pending mark. Nothing is read
// from the map.
__global__ void commit_kernel(MapEntry *map, int64_t n, Ws w, int64_t n_old, int64_t capacity) {
    if (!batch_fits(w, n_old, capacity))
        return;
    for (int64_t i = global_id(); i < n; i += grid_stride()) {
        const int64_t s = w.slot[i];
        if (s < 0)
            continue;
        const bool first = first_new(w, i) != 0, last = w.last[i] != 0;
        const int32_t pos = (int32_t)(n_old + w.rank[i]);
        if (first && last) {
            typedef int pair_t __attribute__((ext_vector_type(2)));
            *reinterpret_cast<pair_t *>(&map[s].pos) = pair_t{pos, -1};
        } else if (first) {
            map[s].pos = pos;
        } else if (last) {
            map[s].aux = -1;
        }
    }
}

unsigned grid_for(int64_t work, int64_t per_block) {
    int64_t b = (work + per_block - 1) / per_block;
    if (b < 1)
        b = 1;
    return (unsigned)(b < 65536 ? b : 65536);
}

__global__ void narrow_kernel(const int64_t *__restrict__ src, int32_t *__restrict__ dst,
                              int64_t n, unsigned long long *wide) {
    unsigned long long local = 0;
    for (int64_t i = global_id(); i < n; i += grid_stride()) {
        const int64_t x = src[i];
        dst[i] = (int32_t)x;
        local += (x < INT32_MIN || x > INT32_MAX) ? 1 : 0;
    }
    if (local)
        atomicAdd(wide, local);
}

// Sets one store counter to zero. A kernel, not a memset: a memset node recorded into a HIP
// graph can leave wrong contents on replays after the first.
__global__ void clear_counter_kernel(unsigned long long *counter) {
    if (threadIdx.x == 0)
        *counter = 0;
}

}  // namespace

hipError_t launch_clear_counter(unsigned long long *counter, hipStream_t stream) {
    hipLaunchKernelGGL(clear_counter_kernel, dim3(1), dim3(64), 0, stream, counter);
    return hipGetLastError();
}

hipError_t launch_narrow_authors(const int64_t *src, int32_t *dst, int64_t n,
                                 unsigned long long *wide, hipStream_t stream) {
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(narrow_kernel, dim3(grid_for(n, kThreads)), dim3(kThreads), 0, stream, src,
                       dst, n, wide);
    return hipGetLastError();
}

int64_t map_groups_for(int64_t capacity) {
    int64_t g = 64;
    while (g * kGroup < 2 * capacity)
        g <<= 1;
    return g;
}

hipError_t launch_map_init(MapEntry *map, int64_t n_groups, hipStream_t stream) {
    const int64_t n = n_groups * kGroup;
    hipLaunchKernelGGL(map_init_kernel, dim3(grid_for(n, kThreads)), dim3(kThreads), 0, stream,
                       map, n);
    return hipGetLastError();
}

hipError_t launch_resolve(const MapEntry *map, int64_t n_groups, const int64_t *ids, int64_t n,
                          int64_t *pos, hipStream_t stream) {
    if (n <= 0)
        return hipSuccess;
    const int64_t quads = (n + kResolvePer - 1) / kResolvePer;
    hipLaunchKernelGGL(resolve_kernel, dim3(grid_for(quads * kGroup, kThreads)), dim3(kThreads), 0,
                       stream, map, (uint64_t)(n_groups - 1), ids, n, pos);
    return hipGetLastError();
}

int64_t upsert_workspace_bytes(int64_t n) {
    if (n <= 0 || n > kMaxBatch)            // the upsert rejects larger batches
        return 0;
    const int64_t blocks = (n + kThreads * kScanPerSmall - 1) / (kThreads * kScanPerSmall);
    return round_up(n * 8) + 2 * round_up(n * 4) + 2 * round_up(n) + round_up(blocks * 8) + 256;
}

int64_t *upsert_counts(void *workspace, int64_t n) { return carve(workspace, n).counts; }

hipError_t launch_upsert_claim(MapEntry *map, int64_t n_groups, const int64_t *ids, int64_t n,
                               void *workspace, int32_t max_polls, hipStream_t stream) {
    const Ws w = carve(workspace, n);
    const uint64_t mask = (uint64_t)(n_groups - 1);
    hipLaunchKernelGGL(counts_init_kernel, dim3(grid_for(round_up(n > 0 ? n : 0) / 16, kThreads)),
                       dim3(kThreads), 0, stream, w, n > 0 ? n : 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || n <= 0)
        return e;
    hipLaunchKernelGGL(claim_kernel, dim3(grid_for(n * kGroup, kThreads)), dim3(kThreads), 0,
                       stream, map, mask, ids, n, w, max_polls);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (scan_per(n) == kScanPerLarge)
        hipLaunchKernelGGL(scan_kernel<kScanPerLarge>, dim3((unsigned)w.blocks), dim3(kThreads), 0,
                           stream, map, n, w, max_polls);
    else
        hipLaunchKernelGGL(scan_kernel<kScanPerSmall>, dim3((unsigned)w.blocks), dim3(kThreads), 0,
                           stream, map, n, w, max_polls);
    return hipGetLastError();
}

hipError_t launch_upsert_finish(MapEntry *map, int64_t n, void *workspace, int64_t n_old,
                                int64_t capacity, const int64_t *author_in, const void *rows_in,
                                int32_t row_bytes, int64_t *author, int32_t *author32,
                                uint8_t *rows, hipStream_t stream) {
    if (n <= 0)
        return hipSuccess;
    const Ws w = carve(workspace, n);
    const int32_t chunks = row_bytes / 16;
    hipLaunchKernelGGL(scatter_kernel, dim3(grid_for(n * chunks, kThreads * kScatterPer)),
                       dim3(kThreads), 0,
                       stream, n, w, n_old, capacity, author_in,
                       static_cast<const chunk_t *>(rows_in), chunks, author, author32,
                       reinterpret_cast<chunk_t *>(rows));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(commit_kernel, dim3(grid_for(n, kThreads)), dim3(kThreads), 0, stream, map,
                       n, w, n_old, capacity);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    // The rollback runs only for a batch that does not fit; otherwise every workgroup returns at
    // once, so a small grid (grid-stride over the records) keeps that no-op launch short.
    hipLaunchKernelGGL(rollback_kernel, dim3(grid_for(n, kThreads * 64)), dim3(kThreads), 0, stream,
                       map, n, w, n_old, capacity);
    return hipGetLastError();
}

}  // namespace ccj
