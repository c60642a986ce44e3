/* Drives every entry point of the CPU oracle on seeded random inputs, for a build with AddressSanitizer
 * and UndefinedBehaviorSanitizer: any out-of-bounds access, use after free, leak or undefined
 * operation in the oracle stops the run with a report.  Returns 0 when every call succeeded. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/pkv_oracle.h"

static uint64_t rng_state = 0x5EED5A17ull;
static uint64_t rnd(void) {                       /* xorshift64* */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 0x2545F4914F6CDD1Dull;
}

static int check(int ok, const char* what) {
    if (!ok) fprintf(stderr, "oracle driver: %s failed\n", what);
    return ok ? 0 : 1;
}

int main(void) {
    int bad = 0;
    uint8_t buf[600], out[32];
    for (uint32_t len = 0; len < sizeof buf; ++len) {          /* every padding boundary */
        for (uint32_t i = 0; i < len; ++i) buf[i] = (uint8_t)rnd();
        orc_sha256(buf, len, out);
    }
    /* descriptors: random names and values, a duplicate name, an empty descriptor */
    for (int trial = 0; trial < 200; ++trial) {
        orc_field f[8];
        uint8_t names[8][12], values[8][40];
        uint32_t n = (uint32_t)(rnd() % 8);
        for (uint32_t i = 0; i < n; ++i) {
            uint32_t nl = (uint32_t)(rnd() % 12), vl = (uint32_t)(rnd() % 40);
            for (uint32_t j = 0; j < nl; ++j) names[i][j] = (uint8_t)('a' + rnd() % 4);
            for (uint32_t j = 0; j < vl; ++j) values[i][j] = (uint8_t)rnd();
            f[i] = (orc_field){names[i], nl, values[i], vl};
        }
        uint64_t need = 0;
        int rc = orc_encode(f, n, NULL, 0, &need);
        if (rc == ORC_OK) {
            uint8_t* enc = (uint8_t*)malloc(need ? need : 1);
            bad += check(orc_encode(f, n, enc, need, &need) == ORC_OK, "encode");
            if (need > 0) orc_encode(f, n, enc, need - 1, &need);   /* a short buffer: writes at most cap bytes */
            free(enc);
            bad += check(orc_digest(f, n, out) == ORC_OK, "digest");
        } else {
            bad += check(rc == ORC_EDUPDIM, "encode duplicate name");
        }
    }
    /* chains: ragged requests (empty, shorter than a block) at several block sizes and thread counts */
    const uint32_t n_req = 37;
    int64_t tok_off[38], key_off[38];
    tok_off[0] = 0;
    for (uint32_t r = 0; r < n_req; ++r) tok_off[r + 1] = tok_off[r] + (int64_t)(rnd() % 90);
    int32_t* tokens = (int32_t*)malloc(sizeof(int32_t) * (size_t)(tok_off[n_req] + 1));
    for (int64_t i = 0; i < tok_off[n_req]; ++i) tokens[i] = (int32_t)rnd();
    uint8_t* digests = (uint8_t*)malloc(16 * n_req);
    for (uint32_t i = 0; i < 16 * n_req; ++i) digests[i] = (uint8_t)rnd();
    const uint32_t blocks[4] = {1, 7, 16, 32};
    for (int bi = 0; bi < 4; ++bi) {
        int64_t n_keys = orc_key_offsets(tok_off, n_req, blocks[bi], key_off);
        uint8_t* keys = (uint8_t*)malloc(16 * (size_t)(n_keys + 1));
        bad += check(orc_derive(tokens, tok_off, n_req, digests, blocks[bi], keys, 1) == ORC_OK, "derive");
        bad += check(orc_derive(tokens, tok_off, n_req, digests, blocks[bi], keys, 3) == ORC_OK, "derive threads");
        /* index: lookup, store, touch, clone, dump, evict; capacity small enough to reach EFULL */
        for (int threads = 1; threads <= 4; threads += 3) {
            orc_index* t = orc_index_new(64);
            orc_index_set_threads(t, threads);
            int32_t* hits = (int32_t*)calloc(n_req, sizeof(int32_t));
            uint64_t* locs = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(n_keys + 1));
            for (int64_t i = 0; i < n_keys; ++i) locs[i] = rnd() >> 3;
            bad += check(orc_lookup(t, keys, key_off, n_req, hits) == ORC_OK, "lookup");
            int rc = orc_store(t, keys, key_off, n_req, hits, locs);
            bad += check(rc == ORC_OK || rc == ORC_EFULL, "store");
            bad += check(orc_lookup_touch(t, keys, key_off, n_req, hits, 2) == ORC_OK, "lookup touch");
            rc = orc_store_touch(t, keys, key_off, n_req, hits, locs, 3);
            bad += check(rc == ORC_OK || rc == ORC_EFULL, "store touch");
            orc_index* c = orc_index_clone(t);
            uint64_t sz = orc_index_size(c);
            uint8_t* dk = (uint8_t*)malloc(16 * (size_t)(sz + 1));
            uint64_t* dl = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(sz + 1));
            uint32_t* de = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(sz + 1));
            orc_index_dump(c, dk, dl);
            orc_index_dump_epochs(c, de);
            orc_evict(c, sz / 2);
            orc_evict(c, 0);
            for (int64_t i = 0; i < n_keys; ++i) locs[i] = (uint64_t)1 << 62;   /* reserved locations */
            memset(hits, 0, n_req * sizeof(int32_t));
            if (n_keys > 0) bad += check(orc_store(t, keys, key_off, n_req, hits, locs) == ORC_ERESERVED,
                                         "reserved location");
            free(dk); free(dl); free(de);
            orc_index_free(c);
            orc_index_free(t);
            free(hits);
            free(locs);
        }
        free(keys);
    }
    /* the threaded sort: one batch above its threshold */
    {
        const uint32_t big = 70000;
        int64_t off[2] = {0, big};
        uint8_t* keys = (uint8_t*)malloc(16 * (size_t)big);
        uint64_t* locs = (uint64_t*)malloc(sizeof(uint64_t) * big);
        for (uint32_t i = 0; i < 16 * big; ++i) keys[i] = (uint8_t)rnd();
        for (uint32_t i = 0; i < big; ++i) locs[i] = i;
        memcpy(keys + 16, keys, 16);                               /* a duplicate across slices */
        int32_t h = 0;
        orc_index* t = orc_index_new(1 << 20);
        orc_index_set_threads(t, 5);
        bad += check(orc_store(t, keys, off, 1, &h, locs) == ORC_OK, "threaded store");
        bad += check(orc_lookup(t, keys, off, 1, &h) == ORC_OK && h == (int32_t)big, "threaded lookup");
        orc_index_free(t);
        free(keys);
        free(locs);
    }
    free(tokens);
    free(digests);
    uint32_t k[64], iv[8];
    orc_sha256_constants(k, iv);
    return bad ? 1 : 0;
}
