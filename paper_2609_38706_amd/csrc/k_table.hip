// k_table.hip -- the shared-tier index in HBM: init, longest-prefix lookup, store of misses,
// rollback, export and eviction to a budget, on gfx950.
//
// Layout (pkv_internal.h): one 32-byte record per slot {claim word, tag, key bytes 8..15, location},
// four slots to a 128-byte bucket.  A key's home bucket is its first eight bytes masked to the bucket
// count; probing continues over the following buckets, wrapping.  A fixed-budget tier adds epochs[capacity] (uint32):
// the epoch of each entry's last use.
//
// Lookup reads whole buckets: a key is present iff some slot on its probe path holds it, and absent
// once the path meets a never-used slot (removed slots have their own claim marker, so paths run
// through them).  Store claims a slot with one 64-bit compare-and-swap on its claim word, then writes
// the slot's tag and, with one 16-byte store, its {key bytes 8..15, location} pair, all inside the
// slot's own 32-byte sector (gfx950 has no 128-bit compare-and-swap):
//   never used or removed --CAS claim word--> claimed, location kEmpty --16-byte store--> published
// A key's path starts in its home bucket at a slot chosen by two bits of the key and continues over
// the bucket's other slots and then the following buckets.  A lane first scans its key's path up to
// the first never-used slot, remembering the first removed slot; it then claims that slot (or the
// never-used one).  A lane that meets a slot claimed with its
// own claim word but not yet published re-reads it until it is, then compares the rest of the key, so
// two lanes inserting one key always meet in the same slot.  Each store call carries its own
// generation, written into the tag of every entry it inserts: a lane that finds its key inserted by
// the same call lowers the location with atomic min (the smallest location of the batch wins), while
// an entry of an earlier call is left untouched.  No pass after the store is needed.
#include "pkv_internal.h"

namespace pkv {
namespace {

using dev::eq4;
using dev::home_bucket;
using dev::key_words;
using dev::KeyWords;
using dev::report;
using dev::slot_holds;
using dev::slot_never_used;

constexpr uint32_t kWaitLimit = 1u << 20;      // re-reads of one claimed slot before giving up

__device__ __forceinline__ bool cas_relaxed(uint64_t* p, uint64_t expected, uint64_t desired) {
    return __hip_atomic_compare_exchange_strong(p, &expected, desired, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void min_relaxed(uint64_t* p, uint64_t v) {
    __hip_atomic_fetch_min(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_relaxed(uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_relaxed(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

// A key's probe path visits its home bucket and then the following buckets (wrapping), each bucket's
// four slots in the order rot, rot + 1, rot + 2, rot + 3 (mod 4), where rot is two bits of the key's
// second half (independent of the home bucket, which the first half gives).  Keys of one bucket so
// spread their first choices over its four slots, and a store's scan meets a free slot after fewer
// reads than when every key starts at the bucket's first slot.  Position p counts along the path
// from the home bucket's first position; path_slot gives the slot at p.
__device__ __forceinline__ uint64_t path_rotation(const KeyWords& kw) { return kw.hi & 3; }
__device__ __forceinline__ uint64_t path_slot(uint64_t p, uint64_t rot) { return (p & ~3ull) | ((p + rot) & 3); }

// Device-coherent 16-byte access to a slot's {key bytes 8..15, location} pair.  The sc1 bit gives
// the same agent-scope coherence that the compiler uses for relaxed agent-scope atomics (the
// access bypasses the non-coherent part of the XCD's L2), for both words in one memory operation.
// The load waits for its own data (vmcnt 0), as the compiler does not track it.  The store does
// not wait: the lane's next memory access is issued at once, so a publishing iteration costs one
// round trip instead of two (c4 store 0.344 -> 0.324 ms).  That is sound because every wait the
// compiler emits after this store in the kernels that use it is a vmcnt(0), which counts the
// untracked store as well (a test compiles k_table.hip and checks this); the s_nop gives the one
// wait state a VALU write to the store's data registers needs after a store of more than 8 bytes.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void load_pair_coherent(const uint64_t* p, uint64_t& hi, uint64_t& loc) {
    u32x4 v;
    asm volatile("global_load_dwordx4 %0, %1, off sc1\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(p) : "memory");
    hi = (static_cast<uint64_t>(v.y) << 32) | v.x;
    loc = (static_cast<uint64_t>(v.w) << 32) | v.z;
}

__device__ __forceinline__ void store_pair_coherent(uint64_t* p, uint64_t hi, uint64_t loc) {
    const u32x4 v = {static_cast<uint32_t>(hi), static_cast<uint32_t>(hi >> 32), static_cast<uint32_t>(loc),
                     static_cast<uint32_t>(loc >> 32)};
    asm volatile("global_store_dwordx4 %0, %1, off sc1\n\ts_nop 0" : : "v"(p), "v"(v) : "memory");
}

// ---- init -------------------------------------------------------------------------------------
// Every slot {kLoEmpty, tag 0, key bytes all ones, kEmpty}: 16-byte units alternate {claim, tag} and
// {key bytes 8..15, location}.
__global__ __launch_bounds__(256) void k_init(uint4* t, uint64_t capacity) {
    const uint64_t n = capacity * 2;                     // 16-byte units: 2 per slot
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t i = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x; i < n; i += stride)
        t[i] = (i & 1) ? make_uint4(~0u, ~0u, ~0u, ~0u) : make_uint4(~0u, ~0u, 0u, 0u);
}

// ---- lookup: one wavefront per request --------------------------------------------------------
// A request's keys are probed in windows, one lane per key; a lane loads its key's bucket (eight
// 16-byte loads issued together: each slot's {claim word, tag} and {key bytes 8..15, location}),
// and the next window's keys are fetched while the current window's buckets are in flight.  A
// ballot finds the first absent key, which ends the request.  The first window holds
// kFirstWindow keys and each later window twice as many, up to 64: probes past a request's first
// miss are wasted bandwidth, so short prefixes (and misses on the first key) probe few keys,
// while long prefixes soon reach full 64-key windows.
constexpr int kLookupWaves = 4;
constexpr uint32_t kFirstWindow = 16;

struct Bucket {
    uint4 c[4];      // slot j: {claim word, tag}
    uint4 p[4];      // slot j: {key bytes 8..15, location}
};

__device__ __forceinline__ void load_bucket(const uint4* __restrict__ t, uint64_t b, Bucket& bk) {
    const uint4* q = t + b * (kBucketWords / 2);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        bk.c[j] = q[2 * j];
        bk.p[j] = q[2 * j + 1];
    }
}

// Probe of one key (lane-private) whose home bucket is already loaded in bk.  Returns the slot
// holding the key, or -1 when it is absent; continues to later buckets while a bucket neither
// matches nor holds a never-used slot.
__device__ __forceinline__ int64_t probe_key(const uint4* __restrict__ t, uint64_t bmask, const uint4& key,
                                             uint64_t b, Bucket& bk) {
    const KeyWords kw = key_words(key);
    const uint64_t n_buckets = bmask + 1;
    for (uint64_t it = 0; it < n_buckets; ++it) {
        bool empty = false;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (slot_holds(bk.c[j], bk.p[j], kw)) return static_cast<int64_t>(b * kSlotsPerBucket + j);
            empty |= slot_never_used(bk.c[j]);
        }
        if (empty) return -1;
        b = (b + 1) & bmask;
        load_bucket(t, b, bk);
    }
    return -1;
}

__global__ __launch_bounds__(64 * kLookupWaves) void k_lookup(const uint4* __restrict__ t, uint64_t capacity,
                                                            const uint4* __restrict__ keys,
                                                            const int64_t* __restrict__ key_off, uint32_t n_req,
                                                            uint64_t n_keys, int32_t* __restrict__ hits,
                                                            uint32_t* epochs, uint32_t epoch, int32_t* status) {
    const uint32_t lane = lane_id();
    const uint32_t r = blockIdx.x * kLookupWaves + (threadIdx.x >> 6);
    if (r >= n_req) return;
    const int64_t k0 = key_off[r], k1 = key_off[r + 1];
    if (k0 < 0 || k1 < k0 || static_cast<uint64_t>(k1) > n_keys) {
        if (lane == 0) {
            report(status, PKV_ELAYOUT);
            hits[r] = 0;
        }
        return;
    }
    const int64_t n = k1 - k0;
    if (n == 0) {
        if (lane == 0) hits[r] = 0;
        return;
    }
    const uint64_t bmask = capacity / kSlotsPerBucket - 1;
    const uint4 marker = make_uint4(~0u, ~0u, ~0u, ~0u);

    // Key idx of the request, or the marker for a lane outside the window or past the request's
    // end (no load is made for those).
    auto key_at = [&](int64_t idx, bool want) {
        if (!want || idx >= n) return marker;
        return keys[k0 + idx];
    };
    int64_t base = 0;
    uint32_t width = kFirstWindow;
    uint4 nk = key_at(lane, lane < width);
    int64_t h = n;
    while (base < n) {
        const uint4 ck = nk;
        const bool v = lane < width && base + lane < n;
        const uint64_t bk = home_bucket(ck, bmask);
        Bucket bucket;
        if (v) load_bucket(t, bk, bucket);
        // next window: twice as wide, up to the wavefront
        const uint32_t next_width = width * 2 < 64 ? width * 2 : 64;
        const int64_t next_base = base + width;
        nk = key_at(next_base + lane, next_base < n && lane < next_width);
        const int64_t fslot = v ? probe_key(t, bmask, ck, bk, bucket) : -1;
        const uint64_t miss = __ballot(v && fslot < 0);
        const int64_t stop = miss ? base + __builtin_ctzll(miss) : -1;
        if (epochs && fslot >= 0 && (stop < 0 || base + lane < stop))   // a touching lookup refreshes hits
            epochs[fslot] = epoch;
        if (stop >= 0) {
            h = stop;
            break;
        }
        base = next_base;
        width = next_width;
    }
    if (lane == 0) hits[r] = static_cast<int32_t>(h < n ? h : n);
}

// ---- store ------------------------------------------------------------------------------------
// One lane per key of the batch; candidate = key j of request r with j >= hits[r].  A wavefront
// covers 64 consecutive keys: one (wave-uniform) search finds the request of its first key, and
// each lane walks forward over the few request boundaries inside the wavefront.  Only candidates
// load their key and location, after that search: a third of the keys of a typical batch lie in hit
// prefixes, and whole wavefronts of them then read nothing but the offsets and hit lengths.
struct StoreArgs {
    Tab t;
    const uint4* keys;
    const int64_t* key_off;
    uint32_t n_req;
    uint64_t n_keys;
    const int32_t* hits;
    const uint64_t* locs;
    uint64_t* new_slots;
    uint64_t* n_new;
    uint32_t* epochs;          // null unless the store refreshes epochs
    uint32_t epoch;
    uint64_t generation;       // this call's generation (tags of the entries it inserts)
    int32_t* status;
};

constexpr uint32_t kStoreThreads = 256;

// The largest r < n_req with key_off[r] <= wave_base (key_off[0] = 0 <= wave_base always): start
// where equal-length requests would put it, widen by doubling steps until [lo, hi) brackets it, then
// bisect (a batch of equal lengths needs two loads instead of log2(n_req)).
__device__ __forceinline__ uint32_t first_request(const StoreArgs& a, uint64_t wave_base, int64_t total) {
    const int64_t wb = static_cast<int64_t>(wave_base);
    const uint64_t n = a.n_req;
    uint64_t lo = 0, hi = n;
    if (total > 0 && n > 2) {
        // single precision and the hardware reciprocal are close enough for a guess: the doubling
        // steps correct it
        uint64_t g = static_cast<uint64_t>(static_cast<float>(wave_base) *
                                           (static_cast<float>(n) * __builtin_amdgcn_rcpf(static_cast<float>(total))));
        if (g >= n) g = n - 1;
        uint64_t step = 1;
        if (a.key_off[g] <= wb) {
            lo = g;
            while (lo + step < n && a.key_off[lo + step] <= wb) { lo += step; step <<= 1; }
            hi = lo + step < n ? lo + step : n;
        } else {
            hi = g;
            while (hi > step && a.key_off[hi - step] > wb) { hi -= step; step <<= 1; }
            lo = hi > step ? hi - step : 0;
        }
    }
    while (hi - lo > 1) {
        const uint64_t mid = (lo + hi) >> 1;
        if (a.key_off[mid] <= wb) lo = mid; else hi = mid;
    }
    return static_cast<uint32_t>(lo);
}

// The probe of a lane's current candidate.
struct StoreProbe {
    KeyWords kw;
    uint64_t want;             // its location
    uint64_t rot;              // path rotation inside each bucket
    uint64_t p;                // path position
    uint64_t first_free;       // position of the first removed slot met while scanning, or ~0
    uint32_t waits;
    bool scanning;             // phase 1: the key may still sit further along its path
};

// The pair of a slot whose claim word matched and whose location word is published.  The pair is
// written by one 16-byte store after the claim; a first half that still reads as the value every
// free slot holds (all ones) is re-read after an acquire fence, in case the read was stale.
__device__ __forceinline__ void read_published_pair(const uint64_t* p, uint64_t& hi, uint64_t& loc) {
    load_pair_coherent(p, hi, loc);
    if (hi == ~0ull && loc != kEmpty) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        load_pair_coherent(p, hi, loc);
    }
}

// Publishes a claimed slot: its tag (generation and substitute flag), then {key bytes 8..15,
// location} with one 16-byte store.  The two stores may land in either order: a reader that sees
// the location published and the tag still 0 waits for the tag.
__device__ __forceinline__ void publish_slot(const Tab& t, uint64_t s, const KeyWords& kw, uint64_t generation,
                                             uint64_t v) {
    store_relaxed(t.tag(s), make_tag(generation, kw.flag));
    store_pair_coherent(t.pair(s), kw.hi, v);
}

__global__ __launch_bounds__(kStoreThreads) void k_store(StoreArgs a) {
    // Beside the next batch's key derivation, a store wavefront that shares a SIMD with one of its
    // round-issuing wavefronts would only get the issue slots that wavefront leaves idle; one level
    // of priority lets the store's short bursts go first.
    __builtin_amdgcn_s_setprio(1);
    __shared__ uint64_t log_slots[kStoreThreads];       // the workgroup's new slots
    __shared__ uint32_t log_n, waves_done;
    const uint32_t lane = lane_id();
    const uint64_t wave_base = static_cast<uint64_t>(blockIdx.x) * kStoreThreads +
                               __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) * 64ull;
    const int64_t total = a.key_off[a.n_req];
    if (total < 0 || static_cast<uint64_t>(total) > a.n_keys) {
        if (blockIdx.x == 0 && threadIdx.x == 0) report(a.status, PKV_ELAYOUT);
        return;
    }
    if (threadIdx.x == 0) {
        log_n = 0;
        waves_done = 0;
    }
    __syncthreads();
    const Tab& t = a.t;
    const uint64_t slot_mask = t.capacity - 1;
    const uint64_t k = wave_base + lane;
    const bool in_batch = static_cast<int64_t>(k) < total;
    bool live = false;
    if (static_cast<int64_t>(wave_base) < total) {
        uint32_t r = first_request(a, wave_base, total);
        if (in_batch) {
            while (r + 1 < a.n_req && a.key_off[r + 1] <= static_cast<int64_t>(k)) ++r;
            const int64_t j = static_cast<int64_t>(k) - a.key_off[r];
            int64_t h = a.hits[r];
            if (h < 0) h = 0;
            live = j >= h;
        }
    }
    // only candidates read their key and location (keys inside a hit prefix are never stored)
    uint4 key = make_uint4(0u, 0u, 0u, 0u);
    uint64_t want = 0;
    if (live) {
        key = a.keys[k];
        want = a.locs[k];
    }
    if (live && want >= PKV_LOC_LIMIT) {
        report(a.status, PKV_ERESERVED);
        live = false;
    }
    StoreProbe st;
    uint64_t p_begin = 0;                                   // where the current phase of the path began
    if (live) {
        st.kw = key_words(key);
        st.want = want;
        st.rot = path_rotation(st.kw);
        st.p = home_bucket(key, (t.capacity / kSlotsPerBucket) - 1) * kSlotsPerBucket;
        st.first_free = ~0ull;
        st.waits = 0;
        st.scanning = true;
        p_begin = st.p;
    }
    // Each pass first runs a tight scan past the slots that need nothing from the lane: slots of
    // other keys, and removed slots while the key may still sit further along its path (the first
    // of those is remembered).  It stops at a never-used slot, at a slot with the lane's own claim
    // word, or, once the lane claims, at a removed slot; the rest of the pass handles that slot.
    // A whole cycle of the path is detected by returning to the position the current phase began at.
    while (live) {
        // a removed slot stops the scan only once the lane claims: compared against this word
        // (while scanning it repeats the never-used marker, which stops the scan anyway)
        const uint64_t stop_word = st.scanning ? kLoEmpty : kLoRemoved;
        uint64_t s = 0, c = 0, at = st.p;
        bool stop = false;
        do {                                                // straight-line body, one exit test
            at = st.p;
            s = path_slot(at, st.rot);
            c = load_relaxed(t.lo(s));
            stop = (c == kLoEmpty) | (c == st.kw.claim) | (c == stop_word);
            if ((c == kLoRemoved) & (st.first_free == ~0ull)) st.first_free = at;   // only while scanning
            st.p = (at + 1) & slot_mask;
        } while (!stop & (st.p != p_begin));                // else a whole cycle of this phase
        if (stop) st.p = at;                                // the slot to act on
        // the slot's word is examined again below: an empty asm keeps the compiler from carrying
        // the loop's comparison results out of it as lane masks merged on every pass
        asm volatile("" : "+v"(c));
        stop = (c == kLoEmpty) | (c == st.kw.claim) | (c == stop_word);
        bool advance = false, done = false, fail = false;
        if (!stop) {                                        // the cycle ended without a slot to act on
            if (st.scanning && st.first_free != ~0ull) {    // claim the first removed slot of the path
                st.scanning = false;
                st.p = p_begin = st.first_free;
            } else {
                report(a.status, PKV_EFULL);
                fail = true;
            }
        } else if (c != st.kw.claim) {                      // never used, or removed while claiming
            bool try_claim = !st.scanning;
            if (st.scanning) {                              // never used: the key is absent
                st.scanning = false;
                if (st.first_free != ~0ull) st.p = p_begin = st.first_free;   // claim the first removed slot on the path instead
                else {
                    p_begin = st.p;
                    try_claim = true;
                }
            }
            if (try_claim && cas_relaxed(t.lo(s), c, st.kw.claim)) {
                publish_slot(t, s, st.kw, a.generation, st.want);
                if (a.epochs) a.epochs[s] = a.epoch;
                log_slots[atomicAdd(&log_n, 1u)] = s | (c == kLoRemoved ? kFromRemoved : 0);
                done = true;
            }                                               // a lost race reads the slot again
        } else {                                            // the lane's own claim word
            uint64_t hi, loc;
            read_published_pair(t.pair(s), hi, loc);
            if (loc == kEmpty) {                            // claimed, not yet published: read it again
                if (++st.waits >= kWaitLimit) { report(a.status, PKV_ESTALL); fail = true; }
            } else if (hi == st.kw.hi) {
                // the tag tells a substitute claim word's key apart and whether this call inserted
                // the entry; it is only needed for those two questions
                const bool need_tag = st.kw.claim == kLoSub || st.want < loc;
                const uint64_t tag = need_tag ? load_relaxed(t.tag(s)) : 0;
                if (need_tag && tag == 0) {                 // published, tag not landed yet: read it again
                    if (++st.waits >= kWaitLimit) { report(a.status, PKV_ESTALL); fail = true; }
                } else if (st.kw.claim != kLoSub || (tag & 3) == st.kw.flag) {
                    if (st.want < loc && (tag >> 2) == a.generation) min_relaxed(t.loc(s), st.want);
                    if (a.epochs) a.epochs[s] = a.epoch;
                    done = true;
                } else {
                    advance = true;
                }
            } else {
                advance = true;
            }
        }
        if (advance) {                                      // another key under the same claim word
            st.p = (st.p + 1) & slot_mask;
            if (st.p == p_begin) {
                if (st.scanning && st.first_free != ~0ull) {
                    st.scanning = false;
                    st.p = p_begin = st.first_free;
                } else {
                    report(a.status, PKV_EFULL);
                    fail = true;
                }
            }
        }
        if (fail || done) live = false;
    }
    // One counter update per workgroup, by its last wavefront to finish: the others leave at once
    // instead of waiting at a barrier (beside other kernels, a workgroup's wavefronts can finish far
    // apart).  The slot log goes out in the order the lanes claimed.
    uint32_t rank = 0;
    if (lane == 0)
        rank = __hip_atomic_fetch_add(&waves_done, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
    rank = __shfl(rank, 0);
    if (rank != kStoreThreads / 64 - 1) return;
    const uint32_t n_log = __hip_atomic_load(&log_n, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
    uint64_t base = 0;
    if (lane == 0 && n_log)
        base = __hip_atomic_fetch_add(a.n_new, static_cast<uint64_t>(n_log), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    base = __shfl(base, 0);
    if (a.new_slots) {
        for (uint32_t i = lane; i < n_log; i += 64) {
            const uint64_t pos = base + i;
            if (pos < a.n_keys) a.new_slots[pos] = log_slots[i];
            else report(a.status, PKV_ELAYOUT);
        }
    }
}

// ---- rollback and export ------------------------------------------------------------------------
// A slot back to a free state: never used, or removed (two 16-byte stores into its 32-byte record).
__device__ __forceinline__ void clear_slot(const Tab& t, uint64_t s, bool removed) {
    const uint32_t m = removed ? 0xFFFFFFFEu : 0xFFFFFFFFu;            // low word of the claim marker
    *reinterpret_cast<uint4*>(t.lo(s)) = make_uint4(m, ~0u, 0u, 0u);   // claim marker, tag 0
    *reinterpret_cast<uint4*>(t.pair(s)) = make_uint4(~0u, ~0u, ~0u, ~0u);   // key bytes 8..15, kEmpty
}

__global__ __launch_bounds__(256) void k_rollback(Tab t, const uint64_t* slots, const uint64_t* n_slots,
                                                  uint64_t max_slots) {
    uint64_t n = *n_slots;
    if (n > max_slots) n = max_slots;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t i = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x; i < n; i += stride) {
        const uint64_t e = slots[i];
        const uint64_t s = e & ~kFromRemoved;
        if (s < t.capacity)                          // the log says how the slot was found: no read
            clear_slot(t, s, (e & kFromRemoved) != 0);
    }
}

__global__ void k_zero_u64(uint64_t* p) { *p = 0; }

// Occupied entry of slot s (< capacity): its key and location, or false.
__device__ __forceinline__ bool slot_entry(const Tab& t, uint64_t s, uint4& key, uint64_t& loc) {
    uint64_t c = *t.lo(s);
    if (c == kLoEmpty || c == kLoRemoved) return false;
    const uint64_t* p = t.pair(s);
    loc = p[1];
    if (loc == kEmpty) return false;
    if (c == kLoSub) {
        const uint64_t f = *t.tag(s) & 3;
        c = f == 1 ? kLoEmpty : (f == 2 ? kLoRemoved : kLoSub);
    }
    const uint64_t hi = p[0];
    key = make_uint4(static_cast<uint32_t>(c), static_cast<uint32_t>(c >> 32), static_cast<uint32_t>(hi),
                     static_cast<uint32_t>(hi >> 32));
    return true;
}

__global__ __launch_bounds__(256) void k_export(Tab t, uint4* out_keys, uint64_t* out_locs, uint64_t* count) {
    const uint32_t lane = lane_id();
    const uint64_t waves = static_cast<uint64_t>(gridDim.x) * (blockDim.x / 64);
    const uint64_t wave = blockIdx.x * static_cast<uint64_t>(blockDim.x / 64) + (threadIdx.x >> 6);
    for (uint64_t base = wave * 64; base < t.capacity; base += waves * 64) {
        const uint64_t s = base + lane;
        uint4 key = make_uint4(0u, 0u, 0u, 0u);
        uint64_t l = 0;
        const bool occ = s < t.capacity && slot_entry(t, s, key, l);
        const uint64_t mask = __ballot(occ);
        if (!mask) continue;
        const uint32_t leader = __builtin_ctzll(mask);
        uint64_t pos = 0;
        if (lane == leader)
            pos = __hip_atomic_fetch_add(count, static_cast<uint64_t>(__popcll(mask)), __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
        pos = __shfl(pos, leader, 64) + __popcll(mask & ((1ull << lane) - 1));
        if (occ) {
            out_keys[pos] = key;
            out_locs[pos] = l;
        }
    }
}

// ---- eviction to a budget (quiescent index) ---------------------------------------------------
// Generational: with E* the smallest epoch such that at most `budget` live entries were last used
// at or after E*, every live entry used before E* is removed (its slot becomes a removed slot).  E* is found by a radix select over the 32-bit
// epochs in three digits (bits 21-31, 10-20, 0-9): per digit, a histogram pass over the index and
// a one-workgroup scan.  Histograms are kept per workgroup in LDS and flushed with one global
// atomic per non-empty bin, so entries that share an epoch do not contend on one address.  The
// work area holds the three histograms and a small control block.
constexpr uint32_t kDigitBins = 2048;
constexpr uint32_t kSelectThreads = 1024;
constexpr uint32_t kHistThreads = 1024;
constexpr uint32_t kHistBlocks = 256;      // one workgroup per CU: one global atomic per hot bin each
__host__ __device__ constexpr int digit_shift(int d) { return d == 0 ? 21 : (d == 1 ? 10 : 0); }
__host__ __device__ constexpr uint32_t digit_bins(int d) { return d == 2 ? 1024u : 2048u; }

struct EvictCtl {
    uint64_t cut;      // E*: entries with epoch < cut are removed (0: none)
    uint64_t above;    // live entries whose selected leading digits exceed the prefix so far
    uint64_t live;     // live entries before the eviction
    uint32_t prefix;   // leading digits selected so far (epoch >> digit_shift of the next digit)
    uint32_t done;     // 1 when nothing has to be removed, or the selection is complete
};

__device__ __forceinline__ EvictCtl* evict_ctl(uint32_t* work) {
    return reinterpret_cast<EvictCtl*>(work + 3 * kDigitBins);
}

__device__ __forceinline__ bool live_slot(const Tab& t, uint64_t s) {
    const uint64_t c = *t.lo(s);
    return c != kLoEmpty && c != kLoRemoved && *t.loc(s) != kEmpty;
}

__global__ __launch_bounds__(256) void k_evict_clear(uint32_t* work, uint64_t* n_evicted) {
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < 3 * kDigitBins; i += gridDim.x * blockDim.x)
        work[i] = 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        EvictCtl* c = evict_ctl(work);
        c->cut = 0;
        c->above = 0;
        c->live = 0;
        c->prefix = 0;
        c->done = 0;
        *n_evicted = 0;
    }
}

// Increment of an LDS histogram aggregated over the wavefront: lanes with equal bins share one
// atomic.  Every lane of the wavefront must call it (the loop is wavefront-uniform).
__device__ __forceinline__ void lds_hist_add(uint32_t* h, bool act, uint32_t bin) {
    uint64_t todo = __ballot(act);
    while (todo) {
        const uint32_t leader = __builtin_ctzll(todo);
        const uint32_t b = __shfl(bin, leader, 64);
        const uint64_t same = __ballot(act && bin == b) & todo;
        if (lane_id() == leader) atomicAdd(h + b, static_cast<uint32_t>(__popcll(same)));
        todo &= ~same;
    }
}

// Histogram of digit d over the live entries whose higher digits equal the selected prefix.
__global__ __launch_bounds__(kHistThreads) void k_evict_hist(Tab t, const uint32_t* epochs, uint32_t* work, int d) {
    __shared__ uint32_t h[kDigitBins];
    const EvictCtl* c = evict_ctl(work);
    if (c->done) return;                       // uniform: the control block is read-only here
    const uint32_t prefix = c->prefix;
    const int shift = digit_shift(d);
    const uint32_t bins = digit_bins(d);
    for (uint32_t i = threadIdx.x; i < kDigitBins; i += blockDim.x) h[i] = 0;
    __syncthreads();
    const uint64_t waves = static_cast<uint64_t>(gridDim.x) * (blockDim.x / 64);
    const uint64_t wave = blockIdx.x * static_cast<uint64_t>(blockDim.x / 64) + (threadIdx.x >> 6);
    for (uint64_t base = wave * 64; base < t.capacity; base += waves * 64) {
        const uint64_t s = base + lane_id();
        bool act = false;
        uint32_t bin = 0;
        if (s < t.capacity && live_slot(t, s)) {
            const uint32_t e = epochs[s];
            const uint32_t high = d == 0 ? 0u : (e >> (shift + (d == 1 ? 11 : 10)));
            act = high == prefix;
            bin = (e >> shift) & (bins - 1);
        }
        lds_hist_add(h, act, bin);
    }
    __syncthreads();
    uint32_t* g = work + d * kDigitBins;
    for (uint32_t i = threadIdx.x; i < bins; i += blockDim.x)
        if (h[i]) atomicAdd(g + i, h[i]);
}

// One workgroup.  With G(b) = above + sum of hist[b'] over b' >= b, finds the largest b with
// G(b) > budget (it exists whenever G(0) > budget) and extends the selected prefix by b.
__global__ __launch_bounds__(kSelectThreads) void k_evict_select(uint32_t* work, uint64_t budget, int d,
                                                                 uint64_t* n_evicted) {
    __shared__ uint64_t part[kSelectThreads];
    __shared__ uint32_t best;
    __shared__ uint64_t total;
    EvictCtl* c = evict_ctl(work);
    if (c->done) return;
    const uint32_t* hist = work + d * kDigitBins;
    const uint32_t bins = digit_bins(d);
    const uint32_t per = bins / kSelectThreads;          // 2 or 1 bins per thread
    const uint32_t t = threadIdx.x;
    uint64_t mine = 0;
    for (uint32_t i = 0; i < per; ++i) mine += hist[t * per + i];
    part[t] = mine;
    if (t == 0) best = 0;          // raised by atomicMax; some thread always finds a bin when not done
    __syncthreads();
    // inclusive suffix sum over threads (log steps): part[t] = sum over u >= t
    for (uint32_t off = 1; off < kSelectThreads; off <<= 1) {
        const uint64_t add = t + off < kSelectThreads ? part[t + off] : 0;
        __syncthreads();
        part[t] += add;
        __syncthreads();
    }
    // the live entries in bins above this thread's range
    const uint64_t above_t = c->above + part[t] - mine;
    if (t == 0) total = c->above + part[0];
    __syncthreads();
    if (d == 0 && t == 0) c->live = total;
    if (d == 0 && total <= budget) {          // everything fits: nothing to remove
        if (t == 0) c->done = 1;
        return;
    }
    uint64_t acc = above_t, before = 0;
    uint32_t found = 0xFFFFFFFFu;
    for (int i = static_cast<int>(per) - 1; i >= 0; --i) {
        const uint64_t prev = acc;
        acc += hist[t * per + i];
        if (acc > budget) { found = t * per + i; before = prev; break; }
    }
    if (found != 0xFFFFFFFFu) atomicMax(&best, found);
    __syncthreads();
    if (found != 0xFFFFFFFFu && found == best) {
        const uint32_t prefix = (c->prefix << (d == 2 ? 10 : 11)) | found;
        if (d < 2) {
            c->prefix = prefix;
            c->above = before;                    // entries above the selected bin
        } else {
            c->cut = static_cast<uint64_t>(prefix) + 1;
            c->done = 1;
            *n_evicted = c->live - before;        // every live entry below the cut
        }
    }
}

__global__ __launch_bounds__(256) void k_evict_apply(Tab t, const uint32_t* epochs, uint32_t* work) {
    const uint64_t cut = evict_ctl(work)->cut;
    if (cut == 0) return;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t s = blockIdx.x * static_cast<uint64_t>(blockDim.x) + threadIdx.x; s < t.capacity; s += stride) {
        if (!live_slot(t, s) || epochs[s] >= cut) continue;
        clear_slot(t, s, true);
    }
}

// ---- hit sums per request group (omission test) -------------------------------------------------
// One workgroup per group: sums[g] = sum of max(hits[r], 0) over r in [group_off[g], group_off[g+1]).
constexpr uint32_t kSumThreads = 256;

__global__ __launch_bounds__(kSumThreads) void k_sum_hits(const int32_t* hits, uint32_t n_req, const int64_t* group_off,
                                                          uint64_t* sums, int32_t* status) {
    __shared__ uint64_t part[kSumThreads / 64];
    const uint32_t g = blockIdx.x;
    const int64_t r0 = group_off[g], r1 = group_off[g + 1];
    const bool ok = r0 >= 0 && r1 >= r0 && r1 <= static_cast<int64_t>(n_req);
    uint64_t acc = 0;
    if (ok) {
        for (int64_t r = r0 + threadIdx.x; r < r1; r += kSumThreads) {
            const int32_t h = hits[r];
            acc += h > 0 ? static_cast<uint64_t>(h) : 0u;
        }
    }
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) acc += __shfl_xor(acc, d, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t total = 0;
#pragma unroll
        for (uint32_t w = 0; w < kSumThreads / 64; ++w) total += part[w];
        sums[g] = ok ? total : 0u;
        if (!ok) report(status, PKV_ELAYOUT);
    }
}

unsigned grid_for(uint64_t items, unsigned threads, unsigned cap_blocks) {
    uint64_t b = (items + threads - 1) / threads;
    if (b < 1) b = 1;
    if (b > cap_blocks) b = cap_blocks;
    return static_cast<unsigned>(b);
}

}  // namespace

int launch_sum_hits(const int32_t* hits, uint32_t n_req, const int64_t* group_off, uint32_t n_groups, uint64_t* sums,
                    int32_t* status, hipStream_t s) {
    if (n_groups == 0) return PKV_OK;
    hipLaunchKernelGGL(k_sum_hits, dim3(n_groups), dim3(kSumThreads), 0, s, hits, n_req, group_off, sums, status);
    return check_launch("pkv_sum_hits");
}

int launch_evict(uint64_t* table, uint64_t capacity, const uint32_t* epochs, uint64_t budget, uint32_t* work,
                 uint64_t* n_evicted, hipStream_t s) {
    const Tab t{table, capacity};
    const unsigned g = grid_for(capacity, kHistThreads, kHistBlocks);
    hipLaunchKernelGGL(k_evict_clear, dim3(8), dim3(256), 0, s, work, n_evicted);
    for (int d = 0; d < 3; ++d) {
        hipLaunchKernelGGL(k_evict_hist, dim3(g), dim3(kHistThreads), 0, s, t, epochs, work, d);
        hipLaunchKernelGGL(k_evict_select, dim3(1), dim3(kSelectThreads), 0, s, work, budget, d, n_evicted);
    }
    hipLaunchKernelGGL(k_evict_apply, dim3(grid_for(capacity, 256, 16384)), dim3(256), 0, s, t, epochs, work);
    return check_launch("pkv_table_evict");
}

int launch_table_init(uint64_t* table, uint64_t capacity, hipStream_t s) {
    hipLaunchKernelGGL(k_init, dim3(grid_for(capacity * 2, 256, 16384)), dim3(256), 0, s,
                       reinterpret_cast<uint4*>(table), capacity);
    return check_launch("pkv_table_init");
}

int launch_lookup(const uint64_t* table, uint64_t capacity, const uint8_t* keys, const int64_t* key_off,
                  uint32_t n_req, uint64_t n_keys, int32_t* hits, uint32_t* epochs, uint32_t epoch, int32_t* status,
                  hipStream_t s) {
    if (n_req == 0) return PKV_OK;
    hipLaunchKernelGGL(k_lookup, dim3((n_req + kLookupWaves - 1) / kLookupWaves), dim3(64 * kLookupWaves), 0, s,
                       reinterpret_cast<const uint4*>(table), capacity, reinterpret_cast<const uint4*>(keys),
                       key_off, n_req, n_keys, hits, epochs, epoch, status);
    return check_launch("pkv_lookup_prefix");
}

int launch_store(uint64_t* table, uint64_t capacity, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
                 uint64_t n_keys, const int32_t* hits, const uint64_t* locs, uint64_t* new_slots, uint64_t* n_new,
                 uint32_t* epochs, uint32_t epoch, int32_t* status, hipStream_t s) {
    if (n_req == 0 || n_keys == 0) return PKV_OK;
    const uint64_t blocks = (n_keys + kStoreThreads - 1) / kStoreThreads;
    if (blocks > 0x7fffffffull) return set_error(PKV_EINVAL, "pkv_store: too many keys (%llu)",
                                                 static_cast<unsigned long long>(n_keys));
    StoreArgs a{Tab{table, capacity}, reinterpret_cast<const uint4*>(keys), key_off, n_req, n_keys, hits, locs,
                new_slots, n_new, epochs, epoch, next_generation(), status};
    hipLaunchKernelGGL(k_store, dim3(static_cast<unsigned>(blocks)), dim3(kStoreThreads), 0, s, a);
    return check_launch("pkv_store");
}

int launch_rollback(uint64_t* table, uint64_t capacity, const uint64_t* slots, const uint64_t* n_slots,
                    uint64_t max_slots, hipStream_t s) {
    if (max_slots == 0) return PKV_OK;
    hipLaunchKernelGGL(k_rollback, dim3(grid_for(max_slots, 256, 8192)), dim3(256), 0, s, Tab{table, capacity}, slots,
                       n_slots, max_slots);
    return check_launch("pkv_table_rollback");
}

int launch_export(const uint64_t* table, uint64_t capacity, uint8_t* out_keys, uint64_t* out_locs, uint64_t* count,
                  hipStream_t s) {
    hipLaunchKernelGGL(k_zero_u64, dim3(1), dim3(1), 0, s, count);
    int rc = check_launch("pkv_table_export (zero)");
    if (rc) return rc;
    const Tab t{const_cast<uint64_t*>(table), capacity};
    hipLaunchKernelGGL(k_export, dim3(grid_for(capacity, 256, 8192)), dim3(256), 0, s, t,
                       reinterpret_cast<uint4*>(out_keys), out_locs, count);
    return check_launch("pkv_table_export");
}

}  // namespace pkv
