// api.cpp -- the C ABI (include/pkv.h): argument checks, the host-side canonical descriptor
// encoder and digest, and the launches of the HIP kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "pkv.h"
#include "pkv_internal.h"

namespace pkv {

namespace {
thread_local char g_error[512] = "no error";

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }
bool pow2(uint64_t x) { return x && !(x & (x - 1)); }

// ---- canonical order (section 5.1 registry, section 5.2 Eq. 3, Prop. 1) -----------------------
constexpr const char* kCoreNames[6] = {"model_id", "adapter_id", "weight_dtype",
                                       "weight_version", "kv_format", "salt"};

struct Ref {
    const pkv_field* f;
    int rank;   // 0..5 core dimension, 6 further dimension
};

int rank_of(const pkv_field& f) {
    for (int i = 0; i < 6; ++i) {
        const size_t n = std::strlen(kCoreNames[i]);
        if (f.name_len == n && std::memcmp(f.name, kCoreNames[i], n) == 0) return i;
    }
    return 6;
}

bool name_less(const pkv_field& a, const pkv_field& b) {
    return std::lexicographical_compare(a.name, a.name + a.name_len, b.name, b.name + b.name_len);
}
bool name_equal(const pkv_field& a, const pkv_field& b) {
    return a.name_len == b.name_len && (a.name_len == 0 || std::memcmp(a.name, b.name, a.name_len) == 0);
}

int canonicalize(const pkv_field* fields, size_t n, std::vector<Ref>& out) {
    out.clear();
    out.reserve(n);
    for (size_t i = 0; i < n; ++i) {
        const pkv_field& f = fields[i];
        if ((f.name_len && !f.name) || (f.value_len && !f.value))
            return set_error(PKV_EINVAL, "pkv_descriptor: field %zu has a null pointer", i);
        out.push_back(Ref{&f, rank_of(f)});
    }
    // unsigned byte order, a proper prefix first (lexicographical_compare on uint8_t)
    std::sort(out.begin(), out.end(), [](const Ref& a, const Ref& b) {
        if (a.rank != b.rank) return a.rank < b.rank;
        return name_less(*a.f, *b.f);
    });
    for (size_t i = 1; i < out.size(); ++i)
        if (name_equal(*out[i].f, *out[i - 1].f))
            return set_error(PKV_EDUPDIM, "pkv_descriptor: dimension name given twice");
    return PKV_OK;
}

void put32(uint8_t* p, uint32_t v) {
    p[0] = static_cast<uint8_t>(v);
    p[1] = static_cast<uint8_t>(v >> 8);
    p[2] = static_cast<uint8_t>(v >> 16);
    p[3] = static_cast<uint8_t>(v >> 24);
}

// ---- host SHA-256 for single descriptors --------------------------------------------------
inline uint32_t hrotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

void host_block(uint32_t st[8], const uint8_t* p) {
    uint32_t w[64];
    for (int t = 0; t < 16; ++t)
        w[t] = (uint32_t(p[4 * t]) << 24) | (uint32_t(p[4 * t + 1]) << 16) | (uint32_t(p[4 * t + 2]) << 8) |
               uint32_t(p[4 * t + 3]);
    for (int t = 16; t < 64; ++t) {
        const uint32_t s0 = hrotr(w[t - 15], 7) ^ hrotr(w[t - 15], 18) ^ (w[t - 15] >> 3);
        const uint32_t s1 = hrotr(w[t - 2], 17) ^ hrotr(w[t - 2], 19) ^ (w[t - 2] >> 10);
        w[t] = w[t - 16] + s0 + w[t - 7] + s1;
    }
    uint32_t v[8];
    std::memcpy(v, st, sizeof v);
    for (int t = 0; t < 64; ++t) {
        const uint32_t e = v[4], a = v[0];
        const uint32_t t1 = v[7] + (hrotr(e, 6) ^ hrotr(e, 11) ^ hrotr(e, 25)) + ((e & v[5]) ^ (~e & v[6])) +
                            kRoundK[t] + w[t];
        const uint32_t t2 = (hrotr(a, 2) ^ hrotr(a, 13) ^ hrotr(a, 22)) + ((a & v[1]) ^ (a & v[2]) ^ (v[1] & v[2]));
        std::memmove(v + 1, v, 7 * sizeof(uint32_t));
        v[4] += t1;
        v[0] = t1 + t2;
    }
    for (int i = 0; i < 8; ++i) st[i] += v[i];
}

void host_sha256(const uint8_t* m, size_t len, uint8_t out[32]) {
    uint32_t st[8];
    std::memcpy(st, kInitH, sizeof st);
    size_t done = 0;
    for (; done + 64 <= len; done += 64) host_block(st, m + done);
    uint8_t tail[128] = {0};
    const size_t rest = len - done;
    std::memcpy(tail, m + done, rest);
    tail[rest] = 0x80;
    const size_t tl = rest < 56 ? 64 : 128;
    const uint64_t bits = static_cast<uint64_t>(len) * 8;
    for (int i = 0; i < 8; ++i) tail[tl - 8 + i] = static_cast<uint8_t>(bits >> (56 - 8 * i));
    host_block(st, tail);
    if (tl == 128) host_block(st, tail + 64);
    for (int i = 0; i < 8; ++i) {
        out[4 * i] = static_cast<uint8_t>(st[i] >> 24);
        out[4 * i + 1] = static_cast<uint8_t>(st[i] >> 16);
        out[4 * i + 2] = static_cast<uint8_t>(st[i] >> 8);
        out[4 * i + 3] = static_cast<uint8_t>(st[i]);
    }
}

void host_digest16(const uint8_t* m, size_t len, uint8_t out[16]) {
    uint8_t full[32];
    host_sha256(m, len, full);
    std::memcpy(out, full, 16);
}

void put64(std::vector<uint8_t>& v, uint64_t x) {
    for (int i = 0; i < 8; ++i) v.push_back(static_cast<uint8_t>(x >> (8 * i)));
}
void put32v(std::vector<uint8_t>& v, uint32_t x) {
    for (int i = 0; i < 4; ++i) v.push_back(static_cast<uint8_t>(x >> (8 * i)));
}
void put_bytes(std::vector<uint8_t>& v, const uint8_t* p, size_t n) { v.insert(v.end(), p, p + n); }

bool bytes_less(const uint8_t* a, size_t na, const uint8_t* b, size_t nb) {
    return std::lexicographical_compare(a, a + na, b, b + nb);
}

int check_table(const pkv_table* t, const char* what) {
    if (!t) return set_error(PKV_EINVAL, "%s: null table", what);
    if (!t->slots) return set_error(PKV_EINVAL, "%s: null table memory", what);
    if (!pow2(t->capacity) || t->capacity < kSlotsPerBucket || t->capacity > (1ull << 56))
        return set_error(PKV_EINVAL, "%s: capacity %llu is not a power of two in [4, 2^56]", what,
                         static_cast<unsigned long long>(t->capacity));
    if (!aligned(t->slots, 128)) return set_error(PKV_EINVAL, "%s: table memory not 128-byte aligned", what);
    return PKV_OK;
}
uint64_t* table_words(const pkv_table* t) { return reinterpret_cast<uint64_t*>(t->slots); }
}  // namespace

int set_error(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
    return code;
}

// Store-call generations: strictly increasing within the process, never 0, starting at a random
// point of a 2^60 range so that two processes writing one index rarely share a generation.
uint64_t next_generation() {
    static std::atomic<uint64_t> counter{[] {
        std::random_device rd;
        const uint64_t seed = (static_cast<uint64_t>(rd()) << 32) ^ rd();
        return (seed & ((1ull << 60) - 1)) | 1ull;
    }()};
    return counter.fetch_add(1, std::memory_order_relaxed) + 1;
}

int check_launch(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(PKV_EHIP, "%s: %s", what, hipGetErrorString(e));
    return PKV_OK;
}

}  // namespace pkv

using namespace pkv;

extern "C" {

const char* pkv_last_error(void) { return g_error; }

const char* pkv_version(void) { return "pkv 0.1 gfx950"; }

int pkv_descriptor_encode(const pkv_field* fields, size_t n, uint8_t* out, size_t cap, size_t* out_len) {
    if (!out_len || (n && !fields)) return set_error(PKV_EINVAL, "pkv_descriptor_encode: null argument");
    if (n > 0xFFFFFFFFull) return set_error(PKV_EINVAL, "pkv_descriptor_encode: too many fields");
    std::vector<Ref> order;
    int rc = canonicalize(fields, n, order);
    if (rc) return rc;
    size_t len = 8;
    for (const Ref& r : order) len += 8 + size_t(r.f->name_len) + size_t(r.f->value_len);
    *out_len = len;
    if (len > cap) return out ? set_error(PKV_EINVAL, "pkv_descriptor_encode: buffer of %zu bytes, need %zu",
                                          cap, len)
                              : PKV_OK;
    if (!out) return set_error(PKV_EINVAL, "pkv_descriptor_encode: null output");
    uint8_t* p = out;
    std::memcpy(p, "PKV1", 4);
    put32(p + 4, static_cast<uint32_t>(n));
    p += 8;
    for (const Ref& r : order) {
        put32(p, r.f->name_len);
        if (r.f->name_len) std::memcpy(p + 4, r.f->name, r.f->name_len);
        p += 4 + r.f->name_len;
        put32(p, r.f->value_len);
        if (r.f->value_len) std::memcpy(p + 4, r.f->value, r.f->value_len);
        p += 4 + r.f->value_len;
    }
    return PKV_OK;
}

int pkv_descriptor_digest(const pkv_field* fields, size_t n, uint8_t out[16]) {
    if (!out) return set_error(PKV_EINVAL, "pkv_descriptor_digest: null output");
    size_t len = 0;
    int rc = pkv_descriptor_encode(fields, n, nullptr, 0, &len);
    if (rc) return rc;
    std::vector<uint8_t> buf(len);
    rc = pkv_descriptor_encode(fields, n, buf.data(), buf.size(), &len);
    if (rc) return rc;
    host_digest16(buf.data(), len, out);
    return PKV_OK;
}

int pkv_digest_batch(const uint8_t* d_bytes, uint64_t n_bytes, const int64_t* d_msg_off, const uint32_t* d_msg_len,
                     uint32_t n_msg, uint8_t* d_digests, int32_t* d_status, hipStream_t stream) {
    if (n_msg == 0) return PKV_OK;
    if ((!d_bytes && n_bytes) || !d_msg_off || !d_msg_len || !d_digests || !d_status)
        return set_error(PKV_EINVAL, "pkv_digest_batch: null argument");
    if (!aligned(d_digests, 16)) return set_error(PKV_EINVAL, "pkv_digest_batch: digests not 16-byte aligned");
    return launch_digest_batch(d_bytes, n_bytes, d_msg_off, d_msg_len, n_msg, d_digests, d_status, stream);
}

int pkv_expand_digests(const uint8_t* d_desc_digests, uint32_t n_desc, const uint32_t* d_desc_idx, uint32_t n_req,
                       uint8_t* d_digests, int32_t* d_status, hipStream_t stream) {
    if (n_req == 0) return PKV_OK;
    if ((!d_desc_digests && n_desc) || !d_desc_idx || !d_digests || !d_status)
        return set_error(PKV_EINVAL, "pkv_expand_digests: null argument");
    if (!aligned(d_desc_digests, 16) || !aligned(d_digests, 16))
        return set_error(PKV_EINVAL, "pkv_expand_digests: digests must be 16-byte aligned");
    return launch_expand_digests(d_desc_digests, n_desc, d_desc_idx, n_req, d_digests, d_status, stream);
}

int pkv_key_offsets(const int64_t* d_tok_off, uint32_t n_req, uint32_t block, int64_t* d_key_off,
                    hipStream_t stream) {
    if (!d_tok_off || !d_key_off) return set_error(PKV_EINVAL, "pkv_key_offsets: null argument");
    if (block == 0) return set_error(PKV_EINVAL, "pkv_key_offsets: block size 0");
    return launch_key_offsets(d_tok_off, n_req, block, d_key_off, stream);
}

int pkv_derive_keys(const int32_t* d_tokens, uint64_t n_tokens, const int64_t* d_tok_off, uint32_t n_req,
                    const uint8_t* d_digests, uint32_t block, const int64_t* d_key_off, uint64_t n_keys,
                    uint8_t* d_keys, int32_t* d_status, hipStream_t stream) {
    if (block == 0) return set_error(PKV_EINVAL, "pkv_derive_keys: block size 0");
    if (n_req == 0) return PKV_OK;
    if ((!d_tokens && n_tokens) || !d_tok_off || !d_digests || !d_key_off || (!d_keys && n_keys) || !d_status)
        return set_error(PKV_EINVAL, "pkv_derive_keys: null argument");
    if (!aligned(d_digests, 16) || !aligned(d_keys, 16))
        return set_error(PKV_EINVAL, "pkv_derive_keys: digests and keys must be 16-byte aligned");
    if (!aligned(d_tokens, 4)) return set_error(PKV_EINVAL, "pkv_derive_keys: tokens not 4-byte aligned");
    return launch_derive(d_tokens, n_tokens, d_tok_off, n_req, d_digests, block, d_key_off, n_keys, d_keys, d_status,
                         stream);
}

int pkv_derive_lookup(const int32_t* d_tokens, uint64_t n_tokens, const int64_t* d_tok_off, uint32_t n_req,
                      const uint8_t* d_digests, uint32_t block, const int64_t* d_key_off, uint64_t n_keys,
                      uint8_t* d_keys, const pkv_table* table, int32_t* d_hit_blocks, int32_t* d_status,
                      hipStream_t stream) {
    int rc = check_table(table, "pkv_derive_lookup");
    if (rc) return rc;
    if (block == 0) return set_error(PKV_EINVAL, "pkv_derive_lookup: block size 0");
    if (n_req == 0) return PKV_OK;
    if ((!d_tokens && n_tokens) || !d_tok_off || !d_digests || !d_key_off || (!d_keys && n_keys) || !d_hit_blocks ||
        !d_status)
        return set_error(PKV_EINVAL, "pkv_derive_lookup: null argument");
    if (!aligned(d_digests, 16) || !aligned(d_keys, 16))
        return set_error(PKV_EINVAL, "pkv_derive_lookup: digests and keys must be 16-byte aligned");
    if (!aligned(d_tokens, 4)) return set_error(PKV_EINVAL, "pkv_derive_lookup: tokens not 4-byte aligned");
    return launch_derive_lookup(d_tokens, n_tokens, d_tok_off, n_req, d_digests, block, d_key_off, n_keys, d_keys,
                                table_words(table), table->capacity, d_hit_blocks, d_status, stream);
}

uint64_t pkv_table_bytes(uint64_t capacity) {
    if (!pow2(capacity) || capacity < kSlotsPerBucket || capacity > (1ull << 56)) return 0;
    return capacity * 32;
}

int pkv_table_init(const pkv_table* table, hipStream_t stream) {
    int rc = check_table(table, "pkv_table_init");
    if (rc) return rc;
    return launch_table_init(table_words(table), table->capacity, stream);
}

int pkv_lookup_prefix(const pkv_table* table, const uint8_t* d_keys, const int64_t* d_key_off, uint32_t n_req,
                      uint64_t n_keys, int32_t* d_hit_blocks, int32_t* d_status, hipStream_t stream) {
    int rc = check_table(table, "pkv_lookup_prefix");
    if (rc) return rc;
    if (n_req == 0) return PKV_OK;
    if ((!d_keys && n_keys) || !d_key_off || !d_hit_blocks || !d_status)
        return set_error(PKV_EINVAL, "pkv_lookup_prefix: null argument");
    if (!aligned(d_keys, 16)) return set_error(PKV_EINVAL, "pkv_lookup_prefix: keys not 16-byte aligned");
    return launch_lookup(table_words(table), table->capacity, d_keys, d_key_off, n_req, n_keys, d_hit_blocks,
                         nullptr, 0, d_status, stream);
}

int pkv_lookup_prefix_touch(const pkv_table* table, const uint8_t* d_keys, const int64_t* d_key_off, uint32_t n_req,
                            uint64_t n_keys, uint32_t* d_epochs, uint32_t epoch, int32_t* d_hit_blocks,
                            int32_t* d_status, hipStream_t stream) {
    int rc = check_table(table, "pkv_lookup_prefix_touch");
    if (rc) return rc;
    if (n_req == 0) return PKV_OK;
    if ((!d_keys && n_keys) || !d_key_off || !d_hit_blocks || !d_status || !d_epochs)
        return set_error(PKV_EINVAL, "pkv_lookup_prefix_touch: null argument");
    if (!aligned(d_keys, 16)) return set_error(PKV_EINVAL, "pkv_lookup_prefix_touch: keys not 16-byte aligned");
    return launch_lookup(table_words(table), table->capacity, d_keys, d_key_off, n_req, n_keys, d_hit_blocks,
                         d_epochs, epoch, d_status, stream);
}

int pkv_store(const pkv_table* table, const uint8_t* d_keys, const int64_t* d_key_off, uint32_t n_req,
              uint64_t n_keys, const int32_t* d_hit_blocks, const uint64_t* d_locs, uint64_t* d_new_slots,
              uint64_t* d_n_new, int32_t* d_status, hipStream_t stream) {
    int rc = check_table(table, "pkv_store");
    if (rc) return rc;
    if (n_req == 0) return PKV_OK;
    if ((!d_keys && n_keys) || !d_key_off || !d_hit_blocks || (!d_locs && n_keys) || !d_n_new || !d_status)
        return set_error(PKV_EINVAL, "pkv_store: null argument");
    if (!aligned(d_keys, 16)) return set_error(PKV_EINVAL, "pkv_store: keys not 16-byte aligned");
    return launch_store(table_words(table), table->capacity, d_keys, d_key_off, n_req, n_keys, d_hit_blocks,
                        d_locs, d_new_slots, d_n_new, nullptr, 0, d_status, stream);
}

int pkv_store_touch(const pkv_table* table, const uint8_t* d_keys, const int64_t* d_key_off, uint32_t n_req,
                    uint64_t n_keys, const int32_t* d_hit_blocks, const uint64_t* d_locs, uint64_t* d_new_slots,
                    uint64_t* d_n_new, uint32_t* d_epochs, uint32_t epoch, int32_t* d_status, hipStream_t stream) {
    int rc = check_table(table, "pkv_store_touch");
    if (rc) return rc;
    if (n_req == 0) return PKV_OK;
    if ((!d_keys && n_keys) || !d_key_off || !d_hit_blocks || (!d_locs && n_keys) || !d_n_new || !d_status ||
        !d_epochs)
        return set_error(PKV_EINVAL, "pkv_store_touch: null argument");
    if (!aligned(d_keys, 16)) return set_error(PKV_EINVAL, "pkv_store_touch: keys not 16-byte aligned");
    return launch_store(table_words(table), table->capacity, d_keys, d_key_off, n_req, n_keys, d_hit_blocks,
                        d_locs, d_new_slots, d_n_new, d_epochs, epoch, d_status, stream);
}

int pkv_table_evict(const pkv_table* table, const uint32_t* d_epochs, uint64_t budget, void* d_work,
                    uint64_t* d_n_evicted, hipStream_t stream) {
    int rc = check_table(table, "pkv_table_evict");
    if (rc) return rc;
    if (!d_epochs || !d_work || !d_n_evicted) return set_error(PKV_EINVAL, "pkv_table_evict: null argument");
    if (!aligned(d_work, 8)) return set_error(PKV_EINVAL, "pkv_table_evict: work area not 8-byte aligned");
    return launch_evict(table_words(table), table->capacity, d_epochs, budget, static_cast<uint32_t*>(d_work),
                        d_n_evicted, stream);
}

int pkv_table_rollback(const pkv_table* table, const uint64_t* d_new_slots, const uint64_t* d_n_new,
                       uint64_t max_slots, hipStream_t stream) {
    int rc = check_table(table, "pkv_table_rollback");
    if (rc) return rc;
    if (max_slots && (!d_new_slots || !d_n_new)) return set_error(PKV_EINVAL, "pkv_table_rollback: null argument");
    return launch_rollback(table_words(table), table->capacity, d_new_slots, d_n_new, max_slots, stream);
}

int pkv_table_export(const pkv_table* table, uint8_t* d_keys_out, uint64_t* d_locs_out, uint64_t* d_count,
                     hipStream_t stream) {
    int rc = check_table(table, "pkv_table_export");
    if (rc) return rc;
    if (!d_keys_out || !d_locs_out || !d_count) return set_error(PKV_EINVAL, "pkv_table_export: null argument");
    if (!aligned(d_keys_out, 16)) return set_error(PKV_EINVAL, "pkv_table_export: output keys not 16-byte aligned");
    return launch_export(table_words(table), table->capacity, d_keys_out, d_locs_out, d_count, stream);
}

int pkv_sum_hits(const int32_t* d_hit_blocks, uint32_t n_req, const int64_t* d_group_off, uint32_t n_groups,
                 uint64_t* d_sums, int32_t* d_status, hipStream_t stream) {
    if (n_groups == 0) return PKV_OK;
    if ((!d_hit_blocks && n_req) || !d_group_off || !d_sums || !d_status)
        return set_error(PKV_EINVAL, "pkv_sum_hits: null argument");
    return launch_sum_hits(d_hit_blocks, n_req, d_group_off, n_groups, d_sums, d_status, stream);
}

uint64_t pkv_tree_work_bytes(uint64_t n_bytes, uint32_t n_tensors) {
    return n_tensors ? tree_layout(n_bytes, n_tensors).bytes : 0;
}

int pkv_tensor_roots(const uint8_t* d_data, uint64_t n_bytes, const int64_t* d_tensor_off, const int64_t* d_tensor_len,
                     uint32_t n_tensors, void* d_work, uint64_t work_bytes, uint8_t* d_roots, int32_t* d_status,
                     hipStream_t stream) {
    if (n_tensors == 0) return PKV_OK;
    if ((!d_data && n_bytes) || !d_tensor_off || !d_tensor_len || !d_work || !d_roots || !d_status)
        return set_error(PKV_EINVAL, "pkv_tensor_roots: null argument");
    if (n_bytes % 4 != 0 || !aligned(d_data, 4))
        return set_error(PKV_EINVAL, "pkv_tensor_roots: data must be 4-byte aligned and a multiple of 4 bytes long");
    if (!aligned(d_work, 256) || !aligned(d_roots, 16))
        return set_error(PKV_EINVAL, "pkv_tensor_roots: work area must be 256-byte and roots 16-byte aligned");
    if (work_bytes < tree_layout(n_bytes, n_tensors).bytes)
        return set_error(PKV_EINVAL, "pkv_tensor_roots: work area smaller than pkv_tree_work_bytes()");
    return launch_tensor_roots(d_data, n_bytes, d_tensor_off, d_tensor_len, n_tensors, static_cast<uint8_t*>(d_work),
                               d_roots, d_status, stream);
}

int pkv_tensor_roots_static(const uint8_t* d_data, uint64_t n_bytes, const int64_t* d_tensor_off,
                            const int64_t* d_tensor_len, uint32_t n_tensors, uint8_t* d_roots, int32_t* d_status,
                            hipStream_t stream) {
    if (n_tensors == 0) return PKV_OK;
    if ((!d_data && n_bytes) || !d_tensor_off || !d_tensor_len || !d_roots || !d_status)
        return set_error(PKV_EINVAL, "pkv_tensor_roots_static: null argument");
    if (n_bytes % 4 != 0 || !aligned(d_data, 4))
        return set_error(PKV_EINVAL, "pkv_tensor_roots_static: data must be 4-byte aligned and a multiple of 4 bytes long");
    if (!aligned(d_roots, 16)) return set_error(PKV_EINVAL, "pkv_tensor_roots_static: roots must be 16-byte aligned");
    const uint64_t need = tree_layout(n_bytes, n_tensors).bytes;
    if (need > PKV_STATIC_TREE_WORK_BYTES)
        return set_error(PKV_EINVAL,
                         "pkv_tensor_roots_static: %llu bytes of data in %u tensors need a %llu-byte work area, more "
                         "than the %llu bytes this entry point holds; use pkv_tensor_roots",
                         static_cast<unsigned long long>(n_bytes), n_tensors, static_cast<unsigned long long>(need),
                         static_cast<unsigned long long>(PKV_STATIC_TREE_WORK_BYTES));
    uint8_t* work = nullptr;
    const int rc = static_tree_work(&work);
    if (rc) return rc;
    return launch_tensor_roots(d_data, n_bytes, d_tensor_off, d_tensor_len, n_tensors, work, d_roots, d_status, stream);
}

int pkv_content_identity(const pkv_tensor* tensors, uint32_t n, const pkv_field* config, size_t n_config,
                         uint8_t out[32]) {
    if ((!tensors && n) || (!config && n_config) || !out) return set_error(PKV_EINVAL, "pkv_content_identity: null argument");
    std::vector<uint32_t> order(n);
    for (uint32_t i = 0; i < n; ++i) {
        const pkv_tensor& t = tensors[i];
        if ((!t.name && t.name_len) || (!t.dtype && t.dtype_len) || (!t.shape && t.ndim) || !t.root)
            return set_error(PKV_EINVAL, "pkv_content_identity: tensor %u has a null field", i);
        order[i] = i;
    }
    std::sort(order.begin(), order.end(), [&](uint32_t a, uint32_t b) {
        return bytes_less(tensors[a].name, tensors[a].name_len, tensors[b].name, tensors[b].name_len);
    });
    for (uint32_t i = 1; i < n; ++i) {
        const pkv_tensor& a = tensors[order[i - 1]];
        const pkv_tensor& b = tensors[order[i]];
        if (a.name_len == b.name_len && (a.name_len == 0 || std::memcmp(a.name, b.name, a.name_len) == 0))
            return set_error(PKV_EDUPDIM, "pkv_content_identity: two tensors share a name");
    }
    std::vector<uint32_t> corder(n_config);
    for (size_t i = 0; i < n_config; ++i) {
        if ((!config[i].name && config[i].name_len) || (!config[i].value && config[i].value_len))
            return set_error(PKV_EINVAL, "pkv_content_identity: configuration field %zu is null", i);
        corder[i] = static_cast<uint32_t>(i);
    }
    std::sort(corder.begin(), corder.end(), [&](uint32_t a, uint32_t b) {
        return bytes_less(config[a].name, config[a].name_len, config[b].name, config[b].name_len);
    });
    for (size_t i = 1; i < n_config; ++i) {
        const pkv_field& a = config[corder[i - 1]];
        const pkv_field& b = config[corder[i]];
        if (a.name_len == b.name_len && (a.name_len == 0 || std::memcmp(a.name, b.name, a.name_len) == 0))
            return set_error(PKV_EDUPDIM, "pkv_content_identity: two configuration fields share a name");
    }
    std::vector<uint8_t> m;
    put_bytes(m, reinterpret_cast<const uint8_t*>("PKVA"), 4);
    put32v(m, n);
    for (uint32_t i : order) {
        const pkv_tensor& t = tensors[i];
        put_bytes(m, reinterpret_cast<const uint8_t*>("PKVT"), 4);
        put32v(m, t.name_len);
        put_bytes(m, t.name, t.name_len);
        put32v(m, t.dtype_len);
        put_bytes(m, t.dtype, t.dtype_len);
        put32v(m, t.ndim);
        for (uint32_t d = 0; d < t.ndim; ++d) put64(m, t.shape[d]);
        put64(m, t.nbytes);
        put_bytes(m, t.root, 32);
    }
    put32v(m, static_cast<uint32_t>(n_config));
    for (uint32_t i : corder) {
        put32v(m, config[i].name_len);
        put_bytes(m, config[i].name, config[i].name_len);
        put32v(m, config[i].value_len);
        put_bytes(m, config[i].value, config[i].value_len);
    }
    host_sha256(m.data(), m.size(), out);
    return PKV_OK;
}

}  // extern "C"
