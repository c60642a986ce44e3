// pkv_internal.h -- shared definitions of the HIP library (device SHA-256, table encoding,
// status reporting, launcher prototypes).  gfx950 only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pkv.h"

namespace pkv {

// FIPS 180-4 section 4.2.2 round constants and section 5.3.3 initial hash value.
static constexpr uint32_t kRoundK[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u, 0x923f82a4u, 0xab1c5ed5u,
    0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u, 0x72be5d74u, 0x80deb1feu, 0x9bdc06a7u, 0xc19bf174u,
    0xe49b69c1u, 0xefbe4786u, 0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu, 0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau,
    0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u, 0xc6e00bf3u, 0xd5a79147u, 0x06ca6351u, 0x14292967u,
    0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu, 0x53380d13u, 0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u,
    0xa2bfe8a1u, 0xa81a664bu, 0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u,
    0x19a4c116u, 0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au, 0x5b9cca4fu, 0x682e6ff3u,
    0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u, 0x90befffau, 0xa4506cebu, 0xbef9a3f7u, 0xc67178f2u};
static constexpr uint32_t kInitH[8] = {0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u, 0xa54ff53au,
                                      0x510e527fu, 0x9b05688cu, 0x1f83d9abu, 0x5be0cd19u};

// Index layout.  One 32-byte record per slot, four consecutive slots to a 128-byte bucket (one HBM
// line), so every access to one slot stays inside one 32-byte sector:
//   word 0  claim word: the key's first 8 bytes (little-endian), or a marker;
//   word 1  tag: (generation << 2) | flag.  The generation is the store call that inserted the
//           entry (every call takes a new one, never 0); the flag says which marker a substitute
//           claim word stands for (1: kLoEmpty, 2: kLoRemoved; 0 for every other key);
//   word 2  key bytes 8..15;
//   word 3  location word.
// Claim word:
//   kLoEmpty    -- never used; ends every probe path through it;
//   kLoRemoved  -- removed by eviction: free for a new key, probe paths continue through it;
//   other       -- claimed by the key whose first 8 bytes it holds.  A key whose first 8 bytes
//                  equal one of the two markers claims with kLoSub instead (and its tag's flag).
// A free slot holds tag 0, key bytes all ones and location kEmpty.  A claimed slot is published
// when its location word (written together with key bytes 8..15 by one 16-byte store) leaves
// kEmpty; its tag is written by a separate store, so a published slot whose tag still reads 0 is
// one whose tag has not landed yet.  Valid caller locations are < 2^62.  Every 128-bit value is an
// ordinary key: the markers live only in claim words, never in key bytes.
static constexpr uint64_t kLoEmpty = ~0ull;
static constexpr uint64_t kLoRemoved = ~0ull - 1;
static constexpr uint64_t kLoSub = ~0ull - 2;
static constexpr uint64_t kEmpty = ~0ull;
static constexpr uint64_t kFromRemoved = 1ull << 63;   // slot-log flag: the claimed slot was a removed entry
static constexpr uint32_t kSlotsPerBucket = 4;
static constexpr uint64_t kSlotWords = 4;           // 32 bytes
static constexpr uint64_t kBucketWords = 16;        // 128 bytes

__host__ __device__ constexpr uint64_t make_tag(uint64_t generation, uint64_t flag) { return (generation << 2) | flag; }

// Word addresses of slot s (< capacity).
struct Tab {
    uint64_t* w;
    uint64_t capacity;
    __device__ __forceinline__ uint64_t* lo(uint64_t s) const { return w + s * kSlotWords; }
    __device__ __forceinline__ uint64_t* tag(uint64_t s) const { return w + s * kSlotWords + 1; }
    __device__ __forceinline__ uint64_t* pair(uint64_t s) const { return w + s * kSlotWords + 2; }
    __device__ __forceinline__ uint64_t* loc(uint64_t s) const { return w + s * kSlotWords + 3; }
};

namespace dev {

__device__ __forceinline__ uint32_t rotr(uint32_t x, uint32_t n) { return __builtin_amdgcn_alignbit(x, x, n); }
// Three-input XOR in one v_bitop3_b32 (truth table 0x96 is symmetric in its inputs).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}
__device__ __forceinline__ uint32_t bsig0(uint32_t a) { return xor3(rotr(a, 2), rotr(a, 13), rotr(a, 22)); }
__device__ __forceinline__ uint32_t bsig1(uint32_t e) { return xor3(rotr(e, 6), rotr(e, 11), rotr(e, 25)); }
__device__ __forceinline__ uint32_t ssig0(uint32_t x) { return xor3(rotr(x, 7), rotr(x, 18), x >> 3); }
__device__ __forceinline__ uint32_t ssig1(uint32_t x) { return xor3(rotr(x, 17), rotr(x, 19), x >> 10); }
__device__ __forceinline__ uint32_t choose(uint32_t e, uint32_t f, uint32_t g) { return g ^ (e & (f ^ g)); }
// Majority in one v_bitop3_b32 (truth table 0xE8 is symmetric in its inputs).
__device__ __forceinline__ uint32_t majority(uint32_t a, uint32_t b, uint32_t c) {
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0xE8);
}
__device__ __forceinline__ uint32_t bswap(uint32_t x) { return __builtin_bswap32(x); }

// One SHA-256 compression (FIPS 180-4 section 6.2.2): s <- s + rounds(s, w).  w holds message
// words 0..15 on entry and is used as the rolling 16-word schedule window.  Fully unrolled, so
// the state rotation is register renaming and the round constants become literals.
__device__ __forceinline__ void compress(uint32_t s[8], uint32_t w[16]) {
    uint32_t a = s[0], b = s[1], c = s[2], d = s[3], e = s[4], f = s[5], g = s[6], h = s[7];
#pragma unroll
    for (int t = 0; t < 64; ++t) {
        uint32_t wt;
        if (t < 16) {
            wt = w[t];
        } else {
            wt = ssig1(w[(t - 2) & 15]) + w[(t - 7) & 15] + ssig0(w[(t - 15) & 15]) + w[t & 15];
            w[t & 15] = wt;
        }
        const uint32_t t1 = h + bsig1(e) + choose(e, f, g) + kRoundK[t] + wt;
        const uint32_t t2 = bsig0(a) + majority(a, b, c);
        h = g; g = f; f = e; e = d + t1;
        d = c; c = b; b = a; a = t1 + t2;
    }
    s[0] += a; s[1] += b; s[2] += c; s[3] += d;
    s[4] += e; s[5] += f; s[6] += g; s[7] += h;
}

__device__ __forceinline__ void init_state(uint32_t s[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) s[i] = kInitH[i];
}

// Records the first device-side error: only a zero status is ever replaced.
__device__ __forceinline__ void report(int32_t* status, int32_t code) {
    int32_t expected = 0;
    __hip_atomic_compare_exchange_strong(status, &expected, code, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool eq4(const uint4& a, const uint4& b) {
    return ((a.x ^ b.x) | (a.y ^ b.y) | (a.z ^ b.z) | (a.w ^ b.w)) == 0;
}

// Home bucket: the key is a SHA-256 output, so its first eight bytes are already uniform.
__device__ __forceinline__ uint64_t home_bucket(const uint4& k, uint64_t bucket_mask) {
    return ((static_cast<uint64_t>(k.y) << 32) | k.x) & bucket_mask;
}

// The two 8-byte halves of a key as little-endian words, and the claim and flag words that stand
// for its first half in a slot.
struct KeyWords {
    uint64_t lo, hi;
    uint64_t claim, flag;
};
__device__ __forceinline__ KeyWords key_words(const uint4& k) {
    KeyWords w;
    w.lo = (static_cast<uint64_t>(k.y) << 32) | k.x;
    w.hi = (static_cast<uint64_t>(k.w) << 32) | k.z;
    w.flag = w.lo == kLoEmpty ? 1u : (w.lo == kLoRemoved ? 2u : 0u);
    w.claim = w.flag ? kLoSub : w.lo;
    return w;
}

// Slot j (0..3) of a bucket as read by a lookup: its {claim word, tag} and {key bytes 8..15,
// location} halves.  The key is in the slot when the claim word (and, under a substitute claim
// word, the flag) and key bytes 8..15 agree and the location is published.
__device__ __forceinline__ bool slot_holds(const uint4& ct, const uint4& pr, const KeyWords& kw) {
    const uint64_t claim = (static_cast<uint64_t>(ct.y) << 32) | ct.x;
    const uint64_t hi = (static_cast<uint64_t>(pr.y) << 32) | pr.x;
    const uint64_t loc = (static_cast<uint64_t>(pr.w) << 32) | pr.z;
    return claim == kw.claim && hi == kw.hi && loc != kEmpty && (kw.claim != kLoSub || (ct.z & 3u) == kw.flag);
}
__device__ __forceinline__ bool slot_never_used(const uint4& ct) {
    return ((static_cast<uint64_t>(ct.y) << 32) | ct.x) == kLoEmpty;
}

}  // namespace dev

// ---- launchers (defined next to their kernels; return a PKV_* code) ------------------------
int launch_digest_batch(const uint8_t* bytes, uint64_t n_bytes, const int64_t* off, const uint32_t* len,
                        uint32_t n, uint8_t* out, int32_t* status, hipStream_t s);
int launch_expand_digests(const uint8_t* desc_digests, uint32_t n_desc, const uint32_t* idx, uint32_t n_req,
                          uint8_t* out, int32_t* status, hipStream_t s);
int launch_key_offsets(const int64_t* tok_off, uint32_t n_req, uint32_t block, int64_t* key_off, hipStream_t s);
int launch_derive(const int32_t* tokens, uint64_t n_tokens, const int64_t* tok_off, uint32_t n_req,
                  const uint8_t* digests, uint32_t block, const int64_t* key_off, uint64_t n_keys,
                  uint8_t* keys, int32_t* status, hipStream_t s);
int launch_table_init(uint64_t* table, uint64_t capacity, hipStream_t s);
int launch_derive_lookup(const int32_t* tokens, uint64_t n_tokens, const int64_t* tok_off, uint32_t n_req,
                         const uint8_t* digests, uint32_t block, const int64_t* key_off, uint64_t n_keys,
                         uint8_t* keys, const uint64_t* table, uint64_t capacity, int32_t* hits, int32_t* status,
                         hipStream_t s);
int launch_lookup(const uint64_t* table, uint64_t capacity, const uint8_t* keys, const int64_t* key_off,
                  uint32_t n_req, uint64_t n_keys, int32_t* hits, uint32_t* epochs, uint32_t epoch, int32_t* status,
                  hipStream_t s);
int launch_store(uint64_t* table, uint64_t capacity, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
                 uint64_t n_keys, const int32_t* hits, const uint64_t* locs, uint64_t* new_slots, uint64_t* n_new,
                 uint32_t* epochs, uint32_t epoch, int32_t* status, hipStream_t s);
uint64_t next_generation();   // a fresh store-call generation (api.hip)
int launch_evict(uint64_t* table, uint64_t capacity, const uint32_t* epochs, uint64_t budget, uint32_t* work,
                 uint64_t* n_evicted, hipStream_t s);
int launch_rollback(uint64_t* table, uint64_t capacity, const uint64_t* slots, const uint64_t* n_slots,
                    uint64_t max_slots, hipStream_t s);
int launch_sum_hits(const int32_t* hits, uint32_t n_req, const int64_t* group_off, uint32_t n_groups, uint64_t* sums,
                    int32_t* status, hipStream_t s);
// Content-identity trees (k_tree.hip).
struct TreeLayout {
    uint32_t levels;
    uint64_t bound[32];        // digests reserved per level
    uint64_t digest_off[32];   // byte offset of each level's digests in the work area
    uint64_t bytes;            // work-area size
};
TreeLayout tree_layout(uint64_t n_bytes, uint32_t n_tensors);
int launch_tensor_roots(const uint8_t* data, uint64_t n_bytes, const int64_t* tensor_off, const int64_t* tensor_len,
                        uint32_t n, uint8_t* work, uint8_t* roots, int32_t* status, hipStream_t s);
int static_tree_work(uint8_t** out);   // device address of the allocation-free entry point's work area
int launch_export(const uint64_t* table, uint64_t capacity, uint8_t* out_keys, uint64_t* out_locs,
                  uint64_t* count, hipStream_t s);

// Host-side error text (api.cpp).
int set_error(int code, const char* fmt, ...);
int check_launch(const char* what);

}  // namespace pkv
