/* pkv_oracle.c -- CPU oracle for provenance-bound KV-cache keys.
 *
 * TEST INFRASTRUCTURE ONLY (see pkv_oracle.h): written for a reader checking it against the
 * paper and FIPS 180-4 by eye, not for speed.  No blocking, no fusion, no reordering beyond
 * what the definitions state.
 */
#include "pkv_oracle.h"

#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------------------------
 * SHA-256, FIPS 180-4.
 * Section 4.2.2: K_t = first 32 bits of the fractional part of the cube root of the t-th prime.
 * Section 5.3.3: H(0)_i = first 32 bits of the fractional part of the square root of the i-th
 * prime.  Both are computed exactly with integer roots of p * 2^96 and p * 2^64.
 * ------------------------------------------------------------------------------------------ */

typedef unsigned __int128 u128;

static uint64_t first_prime(int index) { /* index 0 -> 2 */
    int found = -1;
    for (uint64_t c = 2;; ++c) {
        int is_prime = 1;
        for (uint64_t d = 2; d * d <= c; ++d)
            if (c % d == 0) { is_prime = 0; break; }
        if (is_prime && ++found == index) return c;
    }
}

/* floor(N^(1/e)) for e in {2, 3}, by bisection over [0, 2^40). */
static uint64_t integer_root(u128 n, int e) {
    uint64_t lo = 0, hi = (uint64_t)1 << 40;
    while (hi - lo > 1) {
        uint64_t mid = lo + (hi - lo) / 2;
        u128 p = (u128)mid * mid;
        if (e == 3) p *= mid;
        if (p <= n) lo = mid; else hi = mid;
    }
    return lo;
}

void orc_sha256_constants(uint32_t k[64], uint32_t iv[8]) {
    for (int t = 0; t < 64; ++t) {
        u128 n = (u128)first_prime(t) << 96;             /* cbrt(p * 2^96) = cbrt(p) * 2^32 */
        k[t] = (uint32_t)integer_root(n, 3);              /* keep the fractional 32 bits */
    }
    for (int i = 0; i < 8; ++i) {
        u128 n = (u128)first_prime(i) << 64;             /* sqrt(p * 2^64) = sqrt(p) * 2^32 */
        iv[i] = (uint32_t)integer_root(n, 2);
    }
}

static uint32_t K[64], IV[8];
static pthread_once_t constants_once = PTHREAD_ONCE_INIT;
static void init_constants(void) { orc_sha256_constants(K, IV); }

static uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }
static uint32_t ch(uint32_t x, uint32_t y, uint32_t z) { return (x & y) ^ (~x & z); }
static uint32_t maj(uint32_t x, uint32_t y, uint32_t z) { return (x & y) ^ (x & z) ^ (y & z); }
static uint32_t big_sigma0(uint32_t x) { return rotr(x, 2) ^ rotr(x, 13) ^ rotr(x, 22); }
static uint32_t big_sigma1(uint32_t x) { return rotr(x, 6) ^ rotr(x, 11) ^ rotr(x, 25); }
static uint32_t small_sigma0(uint32_t x) { return rotr(x, 7) ^ rotr(x, 18) ^ (x >> 3); }
static uint32_t small_sigma1(uint32_t x) { return rotr(x, 17) ^ rotr(x, 19) ^ (x >> 10); }

/* FIPS 180-4 section 6.2.2: one 512-bit message block. */
static void compress(uint32_t hash[8], const uint8_t block[64]) {
    uint32_t w[64];
    for (int t = 0; t < 16; ++t)
        w[t] = ((uint32_t)block[4 * t] << 24) | ((uint32_t)block[4 * t + 1] << 16) |
               ((uint32_t)block[4 * t + 2] << 8) | (uint32_t)block[4 * t + 3];
    for (int t = 16; t < 64; ++t)
        w[t] = small_sigma1(w[t - 2]) + w[t - 7] + small_sigma0(w[t - 15]) + w[t - 16];
    uint32_t a = hash[0], b = hash[1], c = hash[2], d = hash[3];
    uint32_t e = hash[4], f = hash[5], g = hash[6], h = hash[7];
    for (int t = 0; t < 64; ++t) {
        uint32_t t1 = h + big_sigma1(e) + ch(e, f, g) + K[t] + w[t];
        uint32_t t2 = big_sigma0(a) + maj(a, b, c);
        h = g; g = f; f = e; e = d + t1;
        d = c; c = b; b = a; a = t1 + t2;
    }
    hash[0] += a; hash[1] += b; hash[2] += c; hash[3] += d;
    hash[4] += e; hash[5] += f; hash[6] += g; hash[7] += h;
}

void orc_sha256(const uint8_t* msg, uint64_t len, uint8_t out[32]) {
    pthread_once(&constants_once, init_constants);
    uint32_t hash[8];
    memcpy(hash, IV, sizeof hash);
    uint64_t full = len / 64;
    for (uint64_t b = 0; b < full; ++b) compress(hash, msg + 64 * b);
    /* Section 5.1.1 padding: a 1 bit, zeros to 448 mod 512 bits, the 64-bit big-endian bit length. */
    uint8_t tail[128];
    memset(tail, 0, sizeof tail);
    uint64_t rest = len - 64 * full;
    memcpy(tail, msg + 64 * full, rest);
    tail[rest] = 0x80;
    uint64_t tail_len = (rest + 1 + 8 <= 64) ? 64 : 128;
    uint64_t bits = len * 8;
    for (int i = 0; i < 8; ++i) tail[tail_len - 1 - i] = (uint8_t)(bits >> (8 * i));
    for (uint64_t off = 0; off < tail_len; off += 64) compress(hash, tail + off);
    for (int i = 0; i < 8; ++i) {
        out[4 * i] = (uint8_t)(hash[i] >> 24);
        out[4 * i + 1] = (uint8_t)(hash[i] >> 16);
        out[4 * i + 2] = (uint8_t)(hash[i] >> 8);
        out[4 * i + 3] = (uint8_t)hash[i];
    }
}

/* H: SHA-256 truncated to its leftmost 128 bits. */
static void trunc_hash(const uint8_t* msg, uint64_t len, uint8_t out[16]) {
    uint8_t full[32];
    orc_sha256(msg, len, full);
    memcpy(out, full, 16);
}

/* ------------------------------------------------------------------------------------------
 * Canonical descriptor encoding (section 5.2, Eq. 3; Prop. 1 appends further dimensions).
 * ------------------------------------------------------------------------------------------ */

static const char* const CORE[6] = {"model_id", "adapter_id", "weight_dtype",
                                    "weight_version", "kv_format", "salt"};

static int core_rank(const orc_field* f) {
    for (int i = 0; i < 6; ++i)
        if (f->name_len == strlen(CORE[i]) && memcmp(f->name, CORE[i], f->name_len) == 0) return i;
    return 6; /* a further registered dimension */
}

static int name_cmp(const orc_field* a, const orc_field* b) {
    uint32_t n = a->name_len < b->name_len ? a->name_len : b->name_len;
    int c = n ? memcmp(a->name, b->name, n) : 0;
    if (c) return c;
    return (a->name_len > b->name_len) - (a->name_len < b->name_len);
}

/* a goes before b in canonical order */
static int canon_before(const orc_field* a, const orc_field* b) {
    int ra = core_rank(a), rb = core_rank(b);
    if (ra != rb) return ra < rb;
    return name_cmp(a, b) < 0;
}

static void put_u32le(uint8_t* p, uint32_t v) {
    p[0] = (uint8_t)v; p[1] = (uint8_t)(v >> 8); p[2] = (uint8_t)(v >> 16); p[3] = (uint8_t)(v >> 24);
}

int orc_encode(const orc_field* f, uint32_t n, uint8_t* out, uint64_t cap, uint64_t* out_len) {
    if ((n && !f) || !out_len) return ORC_EINVAL;
    for (uint32_t i = 0; i < n; ++i)
        for (uint32_t j = i + 1; j < n; ++j)
            if (name_cmp(&f[i], &f[j]) == 0) return ORC_EDUPDIM;
    /* order[] = indices of f in canonical order (insertion sort) */
    uint32_t* order = (uint32_t*)malloc(sizeof(uint32_t) * (n ? n : 1));
    if (!order) return ORC_EINVAL;
    for (uint32_t i = 0; i < n; ++i) {
        uint32_t j = i;
        while (j > 0 && canon_before(&f[i], &f[order[j - 1]])) { order[j] = order[j - 1]; --j; }
        order[j] = i;
    }
    uint64_t len = 4 + 4;
    for (uint32_t i = 0; i < n; ++i) len += 4 + (uint64_t)f[i].name_len + 4 + (uint64_t)f[i].value_len;
    *out_len = len;
    if (out && len <= cap) {
        uint8_t* p = out;
        memcpy(p, "PKV1", 4); p += 4;
        put_u32le(p, n); p += 4;
        for (uint32_t k = 0; k < n; ++k) {
            const orc_field* x = &f[order[k]];
            put_u32le(p, x->name_len); p += 4;
            if (x->name_len) memcpy(p, x->name, x->name_len);
            p += x->name_len;
            put_u32le(p, x->value_len); p += 4;
            if (x->value_len) memcpy(p, x->value, x->value_len);
            p += x->value_len;
        }
    }
    free(order);
    return ORC_OK;
}

int orc_digest(const orc_field* f, uint32_t n, uint8_t out[16]) {
    uint64_t len = 0;
    int rc = orc_encode(f, n, NULL, 0, &len);
    if (rc) return rc;
    uint8_t* buf = (uint8_t*)malloc(len);
    if (!buf) return ORC_EINVAL;
    rc = orc_encode(f, n, buf, len, &len);
    if (rc == ORC_OK) trunc_hash(buf, len, out);
    free(buf);
    return rc;
}

/* ------------------------------------------------------------------------------------------
 * Chained block keys: only complete blocks are keyed (section 4.4: a prefix shorter than one
 * chunk never collides), k_0 = 0^16.
 * ------------------------------------------------------------------------------------------ */

int64_t orc_key_offsets(const int64_t* tok_off, uint32_t n_req, uint32_t block, int64_t* key_off) {
    if (block == 0) return ORC_EINVAL;
    key_off[0] = 0;
    for (uint32_t r = 0; r < n_req; ++r) {
        int64_t len = tok_off[r + 1] - tok_off[r];
        key_off[r + 1] = key_off[r] + len / block;
    }
    return key_off[n_req];
}

static void derive_request(const int32_t* tokens, int64_t len, const uint8_t digest[16],
                           uint32_t block, uint8_t* keys, uint8_t* msg) {
    uint8_t prev[16];
    memset(prev, 0, 16);
    int64_t n = len / block;
    for (int64_t i = 0; i < n; ++i) {
        memcpy(msg, prev, 16);
        memcpy(msg + 16, digest, 16);
        for (uint32_t q = 0; q < block; ++q) {
            uint32_t t = (uint32_t)tokens[i * block + q];
            msg[32 + 4 * q] = (uint8_t)t;
            msg[32 + 4 * q + 1] = (uint8_t)(t >> 8);
            msg[32 + 4 * q + 2] = (uint8_t)(t >> 16);
            msg[32 + 4 * q + 3] = (uint8_t)(t >> 24);
        }
        trunc_hash(msg, 32 + 4 * (uint64_t)block, keys + 16 * i);
        memcpy(prev, keys + 16 * i, 16);
    }
}

typedef struct {
    const int32_t* tokens; const int64_t* tok_off; const uint8_t* digests; uint32_t block;
    uint8_t* keys; const int64_t* key_off; uint32_t r0, r1; int rc;
} derive_job;

static void* derive_worker(void* arg) {
    derive_job* j = (derive_job*)arg;
    uint8_t* msg = (uint8_t*)malloc(32 + 4 * (size_t)j->block);
    if (!msg) { j->rc = ORC_EINVAL; return NULL; }
    for (uint32_t r = j->r0; r < j->r1; ++r)
        derive_request(j->tokens + j->tok_off[r], j->tok_off[r + 1] - j->tok_off[r],
                       j->digests + 16 * (size_t)r, j->block, j->keys + 16 * j->key_off[r], msg);
    free(msg);
    j->rc = ORC_OK;
    return NULL;
}

int orc_derive(const int32_t* tokens, const int64_t* tok_off, uint32_t n_req,
               const uint8_t* digests, uint32_t block, uint8_t* keys, int n_threads) {
    if (block == 0 || n_threads < 1) return ORC_EINVAL;
    pthread_once(&constants_once, init_constants);
    int64_t* key_off = (int64_t*)malloc(sizeof(int64_t) * ((size_t)n_req + 1));
    if (!key_off) return ORC_EINVAL;
    orc_key_offsets(tok_off, n_req, block, key_off);
    if ((uint32_t)n_threads > n_req) n_threads = n_req ? (int)n_req : 1;
    derive_job* jobs = (derive_job*)calloc((size_t)n_threads, sizeof(derive_job));
    pthread_t* th = (pthread_t*)calloc((size_t)n_threads, sizeof(pthread_t));
    int rc = ORC_OK;
    for (int i = 0; i < n_threads; ++i) {
        jobs[i] = (derive_job){tokens, tok_off, digests, block, keys, key_off,
                               (uint32_t)((uint64_t)n_req * i / n_threads),
                               (uint32_t)((uint64_t)n_req * (i + 1) / n_threads), ORC_OK};
        if (n_threads == 1) derive_worker(&jobs[i]);
        else pthread_create(&th[i], NULL, derive_worker, &jobs[i]);
    }
    for (int i = 0; i < n_threads; ++i) {
        if (n_threads > 1) pthread_join(th[i], NULL);
        if (jobs[i].rc) rc = jobs[i].rc;
    }
    free(th); free(jobs); free(key_off);
    return rc;
}

/* ------------------------------------------------------------------------------------------
 * The index as a plain sorted set of (key, location) pairs.
 * ------------------------------------------------------------------------------------------ */

typedef struct { uint8_t key[16]; uint64_t loc; uint32_t epoch; } entry;

/* threads: how many threads the store's sort and the lookup may use (1 by default). */
struct orc_index { uint64_t capacity, size; entry* e; int threads; };

static int entry_cmp(const void* a, const void* b) {
    const entry* x = (const entry*)a; const entry* y = (const entry*)b;
    int c = memcmp(x->key, y->key, 16);
    if (c) return c;
    return (x->loc > y->loc) - (x->loc < y->loc);
}

/* Sorting by entry_cmp on several threads: the array is cut into equal slices, each slice is sorted
 * with qsort on a thread of its own, and neighbouring sorted runs are then merged pairwise (the
 * left run wins ties) until one run is left.  The order is the one a single qsort gives. */
typedef struct { entry* e; uint64_t n; } sort_job;

static void* sort_worker(void* arg) {
    sort_job* j = (sort_job*)arg;
    qsort(j->e, j->n, sizeof(entry), entry_cmp);
    return NULL;
}

static int sort_entries(entry* e, uint64_t n, int threads) {
    if (threads > 64) threads = 64;
    if (threads <= 1 || n < ((uint64_t)1 << 16)) {
        qsort(e, n, sizeof(entry), entry_cmp);
        return ORC_OK;
    }
    uint64_t cut[65];
    for (int i = 0; i <= threads; ++i) cut[i] = n * (uint64_t)i / (uint64_t)threads;
    pthread_t tid[64];
    int running[64];
    sort_job job[64];
    for (int i = 0; i < threads; ++i) {
        job[i].e = e + cut[i];
        job[i].n = cut[i + 1] - cut[i];
        running[i] = pthread_create(&tid[i], NULL, sort_worker, &job[i]) == 0;
        if (!running[i]) sort_worker(&job[i]);           /* no thread: this slice is sorted here */
    }
    for (int i = 0; i < threads; ++i)
        if (running[i]) pthread_join(tid[i], NULL);
    entry* tmp = (entry*)malloc(n * sizeof(entry));
    if (!tmp) return ORC_EINVAL;
    for (int width = 1; width < threads; width *= 2) {
        for (int i = 0; i + width < threads; i += 2 * width) {
            uint64_t lo = cut[i], mid = cut[i + width], hi = cut[i + 2 * width < threads ? i + 2 * width : threads];
            uint64_t a = lo, b = mid, o = 0;
            while (a < mid || b < hi) {
                if (b == hi || (a < mid && entry_cmp(&e[a], &e[b]) <= 0)) tmp[o++] = e[a++];
                else tmp[o++] = e[b++];
            }
            memcpy(e + lo, tmp, (hi - lo) * sizeof(entry));
        }
    }
    free(tmp);
    return ORC_OK;
}

orc_index* orc_index_new(uint64_t capacity) {
    orc_index* t = (orc_index*)calloc(1, sizeof(orc_index));
    if (t) { t->capacity = capacity; t->threads = 1; }
    return t;
}

void orc_index_set_threads(orc_index* t, int threads) { t->threads = threads < 1 ? 1 : threads; }

void orc_index_free(orc_index* t) {
    if (t) { free(t->e); free(t); }
}

orc_index* orc_index_clone(const orc_index* t) {
    orc_index* c = orc_index_new(t->capacity);
    if (!c) return NULL;
    c->threads = t->threads;
    if (t->size) {
        c->e = (entry*)malloc(t->size * sizeof(entry));
        if (!c->e) { free(c); return NULL; }
        memcpy(c->e, t->e, t->size * sizeof(entry));
    }
    c->size = t->size;
    return c;
}

uint64_t orc_index_size(const orc_index* t) { return t->size; }

void orc_index_dump(const orc_index* t, uint8_t* keys, uint64_t* locs) {
    for (uint64_t i = 0; i < t->size; ++i) {
        memcpy(keys + 16 * i, t->e[i].key, 16);
        locs[i] = t->e[i].loc;
    }
}

void orc_index_dump_epochs(const orc_index* t, uint32_t* epochs) {
    for (uint64_t i = 0; i < t->size; ++i) epochs[i] = t->e[i].epoch;
}

/* Position of key in the sorted entries, or -1. */
static int64_t find(const orc_index* t, const uint8_t key[16]) {
    uint64_t lo = 0, hi = t->size;              /* search [lo, hi) */
    while (lo < hi) {
        uint64_t mid = lo + (hi - lo) / 2;
        int c = memcmp(t->e[mid].key, key, 16);
        if (c == 0) return (int64_t)mid;
        if (c < 0) lo = mid + 1; else hi = mid;
    }
    return -1;
}

static int contains(const orc_index* t, const uint8_t key[16]) { return find(t, key) >= 0; }

/* Longest present prefix of requests r0 .. r1 - 1. */
static void lookup_range(const orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t r0, uint32_t r1,
                         int32_t* hits) {
    for (uint32_t r = r0; r < r1; ++r) {
        int64_t n = key_off[r + 1] - key_off[r];
        int64_t h = 0;
        while (h < n && contains(t, keys + 16 * (key_off[r] + h))) ++h;
        hits[r] = (int32_t)h;
    }
}

typedef struct {
    const orc_index* t; const uint8_t* keys; const int64_t* key_off; uint32_t r0, r1; int32_t* hits;
} lookup_job;

static void* lookup_worker(void* arg) {
    lookup_job* j = (lookup_job*)arg;
    lookup_range(j->t, j->keys, j->key_off, j->r0, j->r1, j->hits);
    return NULL;
}

/* The index is only read, so requests are split statically over the index's threads. */
int orc_lookup(const orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
               int32_t* hits) {
    int threads = t->threads > 64 ? 64 : t->threads;
    if (threads <= 1 || n_req < 2) {
        lookup_range(t, keys, key_off, 0, n_req, hits);
        return ORC_OK;
    }
    pthread_t tid[64];
    int running[64];
    lookup_job job[64];
    for (int i = 0; i < threads; ++i) {
        job[i] = (lookup_job){t, keys, key_off, (uint32_t)((uint64_t)n_req * i / threads),
                              (uint32_t)((uint64_t)n_req * (i + 1) / threads), hits};
        running[i] = pthread_create(&tid[i], NULL, lookup_worker, &job[i]) == 0;
        if (!running[i]) lookup_worker(&job[i]);         /* no thread: this slice runs here */
    }
    for (int i = 0; i < threads; ++i)
        if (running[i]) pthread_join(tid[i], NULL);
    return ORC_OK;
}

int orc_lookup_touch(orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
                     int32_t* hits, uint32_t epoch) {
    orc_lookup(t, keys, key_off, n_req, hits);
    for (uint32_t r = 0; r < n_req; ++r)
        for (int64_t j = 0; j < hits[r]; ++j) t->e[find(t, keys + 16 * (key_off[r] + j))].epoch = epoch;
    return ORC_OK;
}

#define ORC_LOC_LIMIT ((uint64_t)1 << 62)

static int store_impl(orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
                      const int32_t* hits, const uint64_t* locs, int touch, uint32_t epoch) {
    /* S = every (k_{r,j}, loc_{r,j}) with j >= h_r */
    uint64_t ns = 0;
    for (uint32_t r = 0; r < n_req; ++r) {
        int64_t n = key_off[r + 1] - key_off[r];
        int64_t h = hits[r] < 0 ? 0 : hits[r];
        if (h < n) ns += (uint64_t)(n - h);
    }
    entry* s = (entry*)malloc(sizeof(entry) * (ns ? ns : 1));
    if (!s) return ORC_EINVAL;
    uint64_t k = 0;
    for (uint32_t r = 0; r < n_req; ++r) {
        int64_t n = key_off[r + 1] - key_off[r];
        for (int64_t j = hits[r] < 0 ? 0 : hits[r]; j < n; ++j) {
            uint64_t idx = (uint64_t)(key_off[r] + j);
            if (locs[idx] >= ORC_LOC_LIMIT) { free(s); return ORC_ERESERVED; }
            memcpy(s[k].key, keys + 16 * idx, 16);
            s[k].loc = locs[idx];
            s[k].epoch = touch ? epoch : 0;
            ++k;
        }
    }
    /* sort by (key, loc): the first of each run of equal keys carries the smallest location */
    if (sort_entries(s, ns, t->threads) != ORC_OK) { free(s); return ORC_EINVAL; }
    uint64_t n_new = 0;
    for (uint64_t i = 0; i < ns; ++i) {
        if (i > 0 && memcmp(s[i].key, s[i - 1].key, 16) == 0) continue;
        if (contains(t, s[i].key)) continue;
        s[n_new++] = s[i];                       /* compact the new keys in place, still sorted */
    }
    /* an index of capacity C holds at most C keys */
    if (t->size + n_new > t->capacity) { free(s); return ORC_EFULL; }
    /* a touching store refreshes the epoch of every candidate key already present */
    if (touch) {
        for (uint32_t r = 0; r < n_req; ++r) {
            int64_t n = key_off[r + 1] - key_off[r];
            for (int64_t j = hits[r] < 0 ? 0 : hits[r]; j < n; ++j) {
                int64_t p = find(t, keys + 16 * (key_off[r] + j));
                if (p >= 0) t->e[p].epoch = epoch;
            }
        }
    }
    /* merge the two sorted runs */
    entry* m = (entry*)malloc(sizeof(entry) * ((t->size + n_new) ? (t->size + n_new) : 1));
    if (!m) { free(s); return ORC_EINVAL; }
    uint64_t a = 0, b = 0, o = 0;
    while (a < t->size || b < n_new) {
        if (b == n_new || (a < t->size && memcmp(t->e[a].key, s[b].key, 16) < 0)) m[o++] = t->e[a++];
        else m[o++] = s[b++];
    }
    free(t->e);
    t->e = m;
    t->size = o;
    free(s);
    return ORC_OK;
}

int orc_store(orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
              const int32_t* hits, const uint64_t* locs) {
    return store_impl(t, keys, key_off, n_req, hits, locs, 0, 0);
}

int orc_store_touch(orc_index* t, const uint8_t* keys, const int64_t* key_off, uint32_t n_req,
                    const int32_t* hits, const uint64_t* locs, uint32_t epoch) {
    return store_impl(t, keys, key_off, n_req, hits, locs, 1, epoch);
}

static int epoch_desc(const void* a, const void* b) {
    uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
    return (x < y) - (x > y);
}

uint64_t orc_evict(orc_index* t, uint64_t budget) {
    if (t->size <= budget) return 0;
    /* E* = smallest E with #{epoch >= E} <= budget = 1 + the (budget+1)-th largest epoch */
    uint32_t* ep = (uint32_t*)malloc(sizeof(uint32_t) * t->size);
    for (uint64_t i = 0; i < t->size; ++i) ep[i] = t->e[i].epoch;
    qsort(ep, t->size, sizeof(uint32_t), epoch_desc);
    uint64_t cut = (uint64_t)ep[budget] + 1;
    free(ep);
    uint64_t o = 0;
    for (uint64_t i = 0; i < t->size; ++i)
        if ((uint64_t)t->e[i].epoch >= cut) t->e[o++] = t->e[i];
    uint64_t evicted = t->size - o;
    t->size = o;
    return evicted;
}
