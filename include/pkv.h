/* pkv.h -- provenance-bound shared-tier KV-cache keys on MI355X (gfx950).
 *
 * C ABI of the hot path of the KV provenance contract (paper section 5): a request's canonical
 * provenance descriptor is encoded and digested (section 5.2, Eq. 3), the digest is folded into
 * chained per-block keys, and the keys probe and then extend a shared-tier index held in HBM.
 *
 *   H(m)       = leftmost 16 bytes of SHA-256(m)                      (FIPS 180-4)
 *   enc(c)     = "PKV1" | u32le(m) | per present field, in canonical order:
 *                u32le(|name|) | name | u32le(|value|) | value         (section 5.2, Eq. 3)
 *   d          = H(enc(c))                                            (the descriptor digest)
 *   key_0      = 16 zero bytes
 *   key_i      = H(key_{i-1} | d | LE32 token ids of block i),  i = 1 .. floor(L / B)
 *   hit_r      = largest h such that key_{r,1..h} are all in the index (a longest-prefix hit)
 *   store      : key_{r,j}, j > hit_r, is inserted if absent; among equal keys of one batch the
 *                smallest location wins; entries already present are never modified
 *                (section 3.4: insert-if-absent, an entry already present is never replaced).
 *
 * Canonical order (section 5.1 registry; Prop. 1 appends further dimensions): the six core
 * dimensions model_id, adapter_id, weight_dtype, weight_version, kv_format, salt in that order,
 * then any further registered dimension by unsigned byte order of its name (a proper prefix
 * first).  An absent dimension is simply not passed, so a request that carries no adapter and
 * no salt keys independently of those two registry entries (section 5.3, request-level tags).
 * Lookup and store take the same key array, so both access sites bind the same descriptor
 * (section 5.3, cross-site consistency).
 *
 * Conventions
 *   - "d_" pointers are device memory owned by the caller; nothing here allocates or frees.
 *   - Device calls are asynchronous on the given stream and never synchronize.  Argument errors
 *     that the host can see are returned synchronously as negative codes (and described by
 *     pkv_last_error()).  Errors found by a kernel (inconsistent offsets, a reserved location, a
 *     full index) are written to the caller's int32 device status word: a kernel only ever
 *     replaces 0 by the first error code it meets, so one zeroed word can serve a whole batch.
 *   - Keys are 16 bytes, stored exactly as the leftmost 16 SHA-256 output bytes.
 *   - Request boundaries are int64 offsets: tokens of request r are tok[tok_off[r] ..
 *     tok_off[r+1]); its keys are keys[key_off[r] .. key_off[r+1]) with key_off[r+1]-key_off[r]
 *     = floor((tok_off[r+1]-tok_off[r]) / B).  A request shorter than one block has no key.
 *   - Locations are caller-defined 64-bit values below PKV_LOC_LIMIT (the top two bits are
 *     reserved for the insert protocol).
 *   - Device errors leave the index contents unspecified.
 *   - Index layout (pkv_table): one device buffer of pkv_table_bytes(capacity) bytes, 128-byte
 *     aligned, capacity a power of two in [4, 2^56].  Slots are indexed 0 .. capacity - 1, and an
 *     index of capacity C holds at most C keys; every 128-bit value is an ordinary key.  A
 *     fixed-budget tier adds an epochs array of capacity uint32.
 */
#ifndef PKV_H
#define PKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    PKV_OK = 0,
    PKV_EINVAL = -1,     /* a malformed argument */
    PKV_EDUPDIM = -2,    /* two descriptor fields share a name */
    PKV_ERESERVED = -3,  /* a location >= PKV_LOC_LIMIT */
    PKV_EFULL = -4,      /* the index has no free slot for a new key */
    PKV_EHIP = -5,       /* a HIP runtime call failed */
    PKV_ELAYOUT = -6,    /* device offsets inconsistent with each other or with buffer sizes */
    PKV_ESTALL = -7,     /* an insert waited too long on a slot another lane had claimed */
};

#define PKV_LOC_LIMIT (1ULL << 62)
#define PKV_KEY_BYTES 16

/* One provenance dimension: its registered name and its identity value, both raw bytes
 * (section 5.1: id_i maps a runtime value to a stable, cross-worker identity). */
typedef struct {
    const uint8_t* name;
    uint32_t name_len;
    const uint8_t* value;
    uint32_t value_len;
} pkv_field;

/* The shared-tier index (section 2.1 shared KV-cache tier): open addressing over buckets of four
 * slots, one 128-byte bucket per HBM line.  Slot s is the 32-byte record at byte 32 s: its claim word
 * (the first 8 key bytes, or a free-slot marker), a tag (the store call that inserted the entry, and
 * which marker a substitute claim word stands for), key bytes 8..15 and the location.  A key's home
 * bucket is its first 8 bytes (little-endian) modulo the bucket count; its probe path visits the
 * home bucket and then the following buckets (wrapping), the slots of each bucket in the order
 * r, r + 1, r + 2, r + 3 (mod 4) with r = key byte 8 mod 4, and a key sits at or before the first
 * never-used slot of its path.
 *   slots    : pkv_table_bytes(capacity) bytes of device memory, 128-byte aligned.
 *   capacity : a power of two in [4, 2^56].
 * The struct itself is host memory; the buffer is device memory owned by the caller. */
typedef struct {
    uint8_t* slots;
    uint64_t capacity;
} pkv_table;
/* Bytes of index memory for `capacity` slots (32 per slot), or 0 when the capacity is not a power
 * of two in [4, 2^56]. */
uint64_t pkv_table_bytes(uint64_t capacity);

/* ---- host, pure, thread-safe ------------------------------------------------------------- */

/* Canonical encoding enc(c) of the n fields (section 5.2, Eq. 3), in any input order.  Writes
 * at most cap bytes to out (out may be NULL when cap is 0); *out_len always receives the full
 * length.  Returns PKV_EDUPDIM if two fields share a name, PKV_EINVAL if out is too small. */
int pkv_descriptor_encode(const pkv_field* fields, size_t n, uint8_t* out, size_t cap, size_t* out_len);

/* d = H(enc(c)) for one descriptor, on the host (the per-request digest of section 6.5). */
int pkv_descriptor_digest(const pkv_field* fields, size_t n, uint8_t out[16]);

/* ---- device, asynchronous on stream ------------------------------------------------------ */

/* Batched descriptor digests on the GPU: d_digests[i] = H(bytes[msg_off[i] .. msg_off[i] +
 * msg_len[i])) for i < n_msg, where each message is a canonical encoding (pkv_descriptor_encode).
 * Messages may overlap, so requests sharing a descriptor can point at one copy.
 * d_bytes: n_bytes bytes.  d_msg_off: n_msg int64.  d_msg_len: n_msg uint32.
 * d_digests: n_msg x 16 bytes, 16-byte aligned.  A message outside [0, n_bytes) sets
 * PKV_ELAYOUT in *d_status and yields no digest. */
int pkv_digest_batch(const uint8_t* d_bytes, uint64_t n_bytes, const int64_t* d_msg_off,
                     const uint32_t* d_msg_len, uint32_t n_msg, uint8_t* d_digests,
                     int32_t* d_status, hipStream_t stream);

/* Per-request digests from per-descriptor digests (section 5.2: one canonical encoder and one
 * digest per descriptor, shared by every request that carries it): d_digests[r] =
 * d_desc_digests[d_desc_idx[r]] for r < n_req.  A batch digests each distinct descriptor once with
 * pkv_digest_batch and expands the results here.  d_desc_digests: n_desc x 16 bytes; d_desc_idx:
 * n_req uint32; d_digests: n_req x 16 bytes; both digest arrays 16-byte aligned.  An index >= n_desc
 * sets PKV_ELAYOUT in *d_status and zeroes that request's digest. */
int pkv_expand_digests(const uint8_t* d_desc_digests, uint32_t n_desc, const uint32_t* d_desc_idx, uint32_t n_req,
                       uint8_t* d_digests, int32_t* d_status, hipStream_t stream);

/* d_key_off[r] = sum over q < r of floor((tok_off[q+1] - tok_off[q]) / block), r = 0..n_req
 * (section 4.4: only complete chunks are keyed).  d_tok_off and d_key_off: n_req + 1 int64.
 * block >= 1.  Offsets must be non-decreasing. */
int pkv_key_offsets(const int64_t* d_tok_off, uint32_t n_req, uint32_t block, int64_t* d_key_off,
                    hipStream_t stream);

/* Chained block keys of n_req requests (section 5.2, Eq. 3 with f = the chained block key).  Beyond
 * the specified (tokens, offsets, digests, block, key offsets, keys) this call takes the token and
 * key counts (bounds checks) and a device status word.
 * d_tokens: n_tokens int32 token ids.  d_tok_off: n_req + 1 int64.  d_digests: n_req x 16
 * bytes (16-byte aligned), one descriptor digest per request.  d_key_off: n_req + 1 int64 as
 * produced by pkv_key_offsets.  d_keys: n_keys x 16 bytes (16-byte aligned).  A request whose
 * offsets fall outside the buffers or disagree with floor(len / block) sets PKV_ELAYOUT and
 * writes no key. */
int pkv_derive_keys(const int32_t* d_tokens, uint64_t n_tokens, const int64_t* d_tok_off,
                    uint32_t n_req, const uint8_t* d_digests, uint32_t block,
                    const int64_t* d_key_off, uint64_t n_keys, uint8_t* d_keys,
                    int32_t* d_status, hipStream_t stream);

/* Chained block keys and their longest-prefix hits in one call (section 5.2, Eq. 3 for the keys;
 * section 3.4 / 4.1 for the hit): the results of pkv_derive_keys followed by pkv_lookup_prefix on
 * the keys it wrote, with the arguments, layouts and errors of those two calls (a request whose
 * offsets are inconsistent gets no key and hit length 0).  For B = 16 and up to two lane-pair
 * workgroups of chains per compute unit (16384 requests on 256 compute units) one kernel does both:
 * each chain's keys are probed while its later keys are still being hashed, so the probes' memory
 * latency hides under the hashing and no key is read back for a separate lookup pass.  Other
 * shapes run the two kernels one after the other.  The index is only read: no store into it may
 * overlap this call (order them on one stream). */
int pkv_derive_lookup(const int32_t* d_tokens, uint64_t n_tokens, const int64_t* d_tok_off, uint32_t n_req,
                      const uint8_t* d_digests, uint32_t block, const int64_t* d_key_off, uint64_t n_keys,
                      uint8_t* d_keys, const pkv_table* table, int32_t* d_hit_blocks, int32_t* d_status,
                      hipStream_t stream);

/* Marks every slot of the index empty: the shared tier starts with no entry (section 2.1 shared
 * KV-cache tier).  Beyond the operations the paper states (digest, derive, lookup, store), the index
 * needs this set-up call, and the export and rollback below. */
int pkv_table_init(const pkv_table* table, hipStream_t stream);

/* Longest-prefix hit per request (section 3.4 / 4.1: the prefix a shared tier can serve; the key
 * count and the device status word are additions to the specified signature):
 * d_hit_blocks[r] = largest h with keys key_off[r] .. key_off[r] + h - 1 all present.
 * d_keys: n_keys x 16 bytes; d_key_off: n_req + 1 int64; d_hit_blocks: n_req int32. */
int pkv_lookup_prefix(const pkv_table* table, const uint8_t* d_keys, const int64_t* d_key_off,
                      uint32_t n_req, uint64_t n_keys, int32_t* d_hit_blocks, int32_t* d_status,
                      hipStream_t stream);

/* Store path (section 2.1: a worker stores the KV blocks it computed into the shared tier;
 * section 3.4: insert-if-absent, an entry already present is never replaced): inserts key j
 * (0-based) of request r with location d_locs[key_off[r] + j] for every j >= d_hit_blocks[r],
 * unless the key is already present.  Duplicates inside the batch keep the smallest location;
 * entries present before the call are never changed.  Compared with the four-call interface the
 * path is specified by, this call also takes the key count (bounds checks), a device status word
 * for errors found by the kernel, an optional slot log (rollback) and a new-entry counter.
 * d_locs: n_keys uint64 (< PKV_LOC_LIMIT, else PKV_ERESERVED).
 * d_n_new: one uint64 counter that the call increments by the number of new entries; the
 * caller zeroes it.  d_new_slots: NULL, or room for n_keys uint64: the slot index of each new
 * entry is appended at d_new_slots[old *d_n_new ...] (bit 63 marks a slot that was removed by
 * eviction before).  No free slot for a new key sets PKV_EFULL.  Calls that store into one index
 * must not overlap in time (order them on one stream). */
int pkv_store(const pkv_table* table, const uint8_t* d_keys, const int64_t* d_key_off,
              uint32_t n_req, uint64_t n_keys, const int32_t* d_hit_blocks, const uint64_t* d_locs,
              uint64_t* d_new_slots, uint64_t* d_n_new, int32_t* d_status, hipStream_t stream);

/* Undoes the stores whose new slots were logged in d_new_slots[0 .. *d_n_new) (at most
 * max_slots), provided nothing else was inserted since: the index returns to its earlier
 * contents exactly.  *d_n_new is left as is. */
int pkv_table_rollback(const pkv_table* table, const uint64_t* d_new_slots, const uint64_t* d_n_new,
                       uint64_t max_slots, hipStream_t stream);

/* Copies every occupied (key, location) pair out, in no particular order: the index contents as
 * a set, which is how stored state is compared with the definition of the store (section 3.4) and
 * how an index is saved across a restart (section 6.3).  d_keys_out: room for
 * capacity keys; d_locs_out: capacity words; *d_count receives the number of pairs (the call
 * zeroes it first). */
int pkv_table_export(const pkv_table* table, uint8_t* d_keys_out, uint64_t* d_locs_out,
                     uint64_t* d_count, hipStream_t stream);

/* Fixed-budget shared tier (section 6.5, eviction under a fixed budget).  Every entry carries
 * the epoch of its last use in d_epochs (capacity uint32, owned by the caller; only entries
 * written through the touching calls have meaningful epochs).
 *
 * pkv_lookup_prefix_touch: pkv_lookup_prefix, and every hit key's epoch becomes `epoch`.
 * pkv_store_touch: pkv_store, and every candidate key (j >= hit length), new or already present,
 * gets epoch `epoch`; present entries keep their locations.  Slots removed by eviction are reused;
 * the slot log marks such a slot with bit 63 so that pkv_table_rollback restores it as removed. */
int pkv_lookup_prefix_touch(const pkv_table* table, const uint8_t* d_keys, const int64_t* d_key_off,
                            uint32_t n_req, uint64_t n_keys, uint32_t* d_epochs, uint32_t epoch,
                            int32_t* d_hit_blocks, int32_t* d_status, hipStream_t stream);
int pkv_store_touch(const pkv_table* table, const uint8_t* d_keys, const int64_t* d_key_off,
                    uint32_t n_req, uint64_t n_keys, const int32_t* d_hit_blocks, const uint64_t* d_locs,
                    uint64_t* d_new_slots, uint64_t* d_n_new, uint32_t* d_epochs, uint32_t epoch,
                    int32_t* d_status, hipStream_t stream);

/* Generational eviction to a budget: with E* the smallest epoch such that at most `budget`
 * entries were last used at or after E*, every entry used before E* is removed (probe paths
 * stay intact: its slot is marked removed, not empty).  d_work: PKV_EVICT_WORK_BYTES of device
 * memory (8-byte aligned, contents overwritten); *d_n_evicted receives the number removed.  The
 * index must not be accessed by other calls while this runs (stream order suffices). */
#define PKV_EVICT_WORK_BYTES ((size_t)(3 * 2048 * 4 + 64))
int pkv_table_evict(const pkv_table* table, const uint32_t* d_epochs, uint64_t budget, void* d_work,
                    uint64_t* d_n_evicted, hipStream_t stream);

/* Store-side form of the differential omission test (section 5.4, Eq. 4; section 6.4 omission
 * detection).  The keys of base configurations are stored, the keys of configurations that differ
 * from them in one dimension are looked up, and a key found is a key the two configurations
 * share.  This call sums the hit lengths per group of requests:
 *   d_sums[g] = sum of max(d_hit_blocks[r], 0) over r in [d_group_off[g], d_group_off[g+1]).
 * d_hit_blocks: n_req int32 (as written by pkv_lookup_prefix); d_group_off: n_groups + 1 int64,
 * non-decreasing, within [0, n_req]; d_sums: n_groups uint64.  A group whose bounds are
 * inconsistent gets 0 and sets PKV_ELAYOUT. */
int pkv_sum_hits(const int32_t* d_hit_blocks, uint32_t n_req, const int64_t* d_group_off, uint32_t n_groups,
                 uint64_t* d_sums, int32_t* d_status, hipStream_t stream);

/* Content identity of an adapter or checkpoint (section 5.3: the adapter is bound by an identity
 * of its contents, every tensor's name, dtype, shape and bytes with the meaningful configuration
 * fields; section 6.5: its cost).  The paper fixes no hash; this library defines:
 *   tensor root : Merkle tree over the tensor's bytes; leaves of 1024 bytes, leaf = SHA-256(0x00 |
 *                 bytes) (an empty tensor has one empty leaf); node = SHA-256(0x01 | up to 16
 *                 consecutive child digests); the first level with one digest holds the root;
 *   record      : "PKVT" | u32(|name|) name | u32(|dtype|) dtype | u32(ndim) u64(dim)... |
 *                 u64(byte length) | root                      (integers little-endian);
 *   identity    : SHA-256("PKVA" | u32(#tensors) | records in name order | u32(#fields) |
 *                 (u32(|key|) key u32(|value|) value)... in key order)       (32 bytes).
 *
 * pkv_tensor_roots (device): the roots of n_tensors tensors whose bytes lie in d_data (n_bytes, a
 * multiple of 4, 4-byte aligned); tensor t occupies [d_tensor_off[t], d_tensor_off[t] +
 * d_tensor_len[t]) (int64; every start a multiple of 4).  Tensors may leave gaps and may overlap,
 * provided their lengths add up to at most n_bytes: the work area is sized for that.
 * d_work: pkv_tree_work_bytes(n_bytes, n_tensors) bytes, 256-byte aligned; d_roots: n_tensors x 32
 * bytes.  A tensor outside the data, or lengths that add up to more than n_bytes, set PKV_ELAYOUT;
 * the roots are then unspecified, and nothing outside d_work and d_roots is written.
 * pkv_content_identity (host, pure): the identity from the tensors' metadata and roots;
 * duplicate tensor names or configuration keys are PKV_EDUPDIM. */
typedef struct {
    const uint8_t* name;
    uint32_t name_len;
    const uint8_t* dtype;
    uint32_t dtype_len;
    const uint64_t* shape;
    uint32_t ndim;
    uint64_t nbytes;
    const uint8_t* root;       /* 32 bytes */
} pkv_tensor;
uint64_t pkv_tree_work_bytes(uint64_t n_bytes, uint32_t n_tensors);
int pkv_tensor_roots(const uint8_t* d_data, uint64_t n_bytes, const int64_t* d_tensor_off, const int64_t* d_tensor_len,
                     uint32_t n_tensors, void* d_work, uint64_t work_bytes, uint8_t* d_roots, int32_t* d_status,
                     hipStream_t stream);
int pkv_content_identity(const pkv_tensor* tensors, uint32_t n_tensors, const pkv_field* config, size_t n_config,
                         uint8_t out[32]);

/* pkv_tensor_roots for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same roots, with the work area taken
 * from a buffer of PKV_STATIC_TREE_WORK_BYTES that the library holds on each device it runs on
 * until the process ends, so the caller passes only inputs and outputs.  The call allocates
 * nothing (no hipMalloc, no hipFree).  Inputs whose work area, pkv_tree_work_bytes(n_bytes,
 * n_tensors), exceeds PKV_STATIC_TREE_WORK_BYTES (about 250 MB of tensor bytes) are refused with
 * PKV_EINVAL before anything is launched.  Every call on one device uses that device's one buffer:
 * calls that overlap on one device (concurrent streams, or threads) race and give unspecified
 * roots; calls ordered on one stream do not.  The first call on a device looks the buffer's address
 * up there (and may return PKV_EHIP if that fails). */
#define PKV_STATIC_TREE_WORK_BYTES (8u << 20)
int pkv_tensor_roots_static(const uint8_t* d_data, uint64_t n_bytes, const int64_t* d_tensor_off,
                            const int64_t* d_tensor_len, uint32_t n_tensors, uint8_t* d_roots, int32_t* d_status,
                            hipStream_t stream);

/* Text describing the last non-OK return on this thread. */
const char* pkv_last_error(void);

/* Library version string. */
const char* pkv_version(void);

#ifdef __cplusplus
}
#endif
#endif
