/* pkv_oracle.h -- CPU oracle for provenance-bound KV-cache keys.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously-correct statement of what the
 * hot path computes.  It is compiled as its own shared library, shares no source, header, table
 * or helper with the product library, and only the tests, the smoke check and the benchmark's
 * CPU-baseline leg may load it.  The product never calls it.
 *
 * What it computes (paper section 5.2, Eq. 3 and Prop. 1; section 5.3 cross-site consistency):
 *   H(m)   = first 16 bytes of SHA-256(m)                      (FIPS 180-4)
 *   enc(c) = "PKV1" | u32le(m) | for each present field in canonical order:
 *            u32le(|name|) | name | u32le(|value|) | value     (injective, length-prefixed)
 *   d      = H(enc(c))                                         (descriptor digest)
 *   k_0    = 16 zero bytes
 *   k_i    = H(k_{i-1} | d | LE32(t_{(i-1)B}) .. LE32(t_{iB-1}))   for i = 1 .. floor(L/B)
 *   lookup: h_r = largest h with k_{r,1..h} all in the index
 *   store:  every k_{r,j}, j > h_r, absent from the index is inserted once; among duplicates in
 *           one batch the smallest location wins; entries already present are never changed.
 *   capacity: an index of capacity C holds at most C keys; a store whose new keys would exceed
 *           that fails as a whole.
 *
 * Canonical order: the six core dimensions first, in the fixed registry order
 *   model_id, adapter_id, weight_dtype, weight_version, kv_format, salt,
 * then every further dimension by unsigned byte order of its name (a proper prefix first).
 * Absent dimensions are simply not passed.  Two fields with the same name are an error.
 */
#ifndef PKV_ORACLE_H
#define PKV_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    ORC_OK = 0,
    ORC_EINVAL = -1,     /* malformed arguments */
    ORC_EDUPDIM = -2,    /* two fields share a name */
    ORC_ERESERVED = -3,  /* a location uses the reserved top two bits */
    ORC_EFULL = -4,      /* the index cannot hold every new key */
};

typedef struct {
    const uint8_t* name;
    uint32_t name_len;
    const uint8_t* value;
    uint32_t value_len;
} orc_field;

/* FIPS 180-4 SHA-256 of len bytes; writes 32 bytes. */
void orc_sha256(const uint8_t* msg, uint64_t len, uint8_t out[32]);

/* The 64 round constants and 8 initial hash words, derived from the first primes. */
void orc_sha256_constants(uint32_t k[64], uint32_t iv[8]);

/* Canonical encoding.  Writes at most cap bytes; *out_len receives the full length. */
int orc_encode(const orc_field* f, uint32_t n, uint8_t* out, uint64_t cap, uint64_t* out_len);

/* d = H(enc(fields)). */
int orc_digest(const orc_field* f, uint32_t n, uint8_t out[16]);

/* key_off[r] = sum over q < r of floor(len_q / block); returns the total key count. */
int64_t orc_key_offsets(const int64_t* tok_off, uint32_t n_req, uint32_t block, int64_t* key_off);

/* Derives every block key of every request (layout given by orc_key_offsets), 16 bytes each.
 * digests holds 16 bytes per request.  n_threads >= 1 splits requests statically. */
int orc_derive(const int32_t* tokens, const int64_t* tok_off, uint32_t n_req,
               const uint8_t* digests, uint32_t block, uint8_t* keys, int n_threads);

/* The index: a set of (key, location) pairs, kept sorted by key. */
typedef struct orc_index orc_index;

orc_index* orc_index_new(uint64_t capacity);
void orc_index_free(orc_index* t);
/* Threads the index's store (its sort) and lookup may use; 1 by default.  Results do not depend
 * on it. */
void orc_index_set_threads(orc_index* t, int threads);
/* An independent copy of t (same capacity, pairs and thread count); NULL if out of memory. */
orc_index* orc_index_clone(const orc_index* t);
uint64_t orc_index_size(const orc_index* t);
/* Copies the pairs out in ascending key order (byte-wise unsigned comparison). */
void orc_index_dump(const orc_index* t, uint8_t* keys, uint64_t* locs);
/* The epochs of the pairs, in the same order. */
void orc_index_dump_epochs(const orc_index* t, uint32_t* epochs);

int orc_lookup(const orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
               int32_t* hits);

/* Inserts every key k_{r,j} with j >= hits[r] (0-based) that the index lacks.  On ORC_EFULL
 * or ORC_ERESERVED the index is left unchanged.  ORC_EFULL: the index would hold more keys than
 * its capacity. */
int orc_store(orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
              const int32_t* hits, const uint64_t* locs);

/* Fixed-budget tier (section 6.5).  Every pair carries the epoch of its last use.  The touching
 * lookup sets the epoch of every hit key to `epoch`; the touching store inserts like orc_store
 * with new pairs at `epoch` and sets the epoch of every candidate key already present. */
int orc_lookup_touch(orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
                     int32_t* hits, uint32_t epoch);
int orc_store_touch(orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
                    const int32_t* hits, const uint64_t* locs, uint32_t epoch);
/* Generational eviction to a budget: with E* the smallest epoch such that at most `budget`
 * pairs have epoch >= E*, removes every pair older than E*.  Returns the number removed. */
uint64_t orc_evict(orc_index* t, uint64_t budget);

#ifdef __cplusplus
}
#endif
#endif
