// Drives the host-side code of the pkv library (canonical encoding, descriptor digest, content
// identity, size queries and the synchronous argument checks of the device calls) on seeded random
// inputs, for a build with AddressSanitizer and UndefinedBehaviorSanitizer on the host code.  No call
// here reaches the GPU.  Returns 0 when every call behaved as the header states.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "pkv.h"

namespace {
uint64_t state = 0x5EEDC0DEull;
uint64_t rnd() {
    state ^= state >> 12;
    state ^= state << 25;
    state ^= state >> 27;
    return state * 0x2545F4914F6CDD1Dull;
}
int bad = 0;
void check(bool ok, const char* what) {
    if (!ok) {
        std::fprintf(stderr, "host driver: %s failed (%s)\n", what, pkv_last_error());
        ++bad;
    }
}
}  // namespace

int main() {
    const char* core[] = {"model_id", "adapter_id", "weight_dtype", "weight_version", "kv_format", "salt"};
    for (int trial = 0; trial < 300; ++trial) {
        const size_t n = rnd() % 9;
        std::vector<std::vector<uint8_t>> names(n), values(n);
        std::vector<pkv_field> f(n);
        for (size_t i = 0; i < n; ++i) {
            if (rnd() % 3 == 0) {
                const char* c = core[rnd() % 6];
                names[i].assign(c, c + std::strlen(c));
            } else {
                names[i].resize(rnd() % 10);
                for (auto& b : names[i]) b = static_cast<uint8_t>('a' + rnd() % 3);
            }
            values[i].resize(rnd() % 50);
            for (auto& b : values[i]) b = static_cast<uint8_t>(rnd());
            f[i] = pkv_field{names[i].data(), static_cast<uint32_t>(names[i].size()), values[i].data(),
                             static_cast<uint32_t>(values[i].size())};
        }
        size_t need = 0;
        const int rc = pkv_descriptor_encode(f.data(), n, nullptr, 0, &need);
        uint8_t d[16];
        if (rc == PKV_OK) {
            std::vector<uint8_t> enc(need + 1);
            check(pkv_descriptor_encode(f.data(), n, enc.data(), need, &need) == PKV_OK, "encode");
            check(pkv_descriptor_encode(f.data(), n, enc.data(), need - 1, &need) == PKV_EINVAL, "encode short buffer");
            check(pkv_descriptor_digest(f.data(), n, d) == PKV_OK, "digest");
        } else {
            check(rc == PKV_EDUPDIM, "encode duplicate name");
            check(pkv_descriptor_digest(f.data(), n, d) == PKV_EDUPDIM, "digest duplicate name");
        }
        // content identity over random tensor records and configuration fields
        const uint32_t nt = static_cast<uint32_t>(rnd() % 6);
        std::vector<pkv_tensor> ts(nt);
        std::vector<std::vector<uint8_t>> tnames(nt);
        std::vector<std::vector<uint64_t>> shapes(nt);
        uint8_t root[32] = {1};
        for (uint32_t i = 0; i < nt; ++i) {
            tnames[i].resize(1 + rnd() % 12);
            for (auto& b : tnames[i]) b = static_cast<uint8_t>('a' + rnd() % 26);
            shapes[i].resize(rnd() % 4);
            for (auto& s : shapes[i]) s = rnd() % 4096;
            ts[i] = pkv_tensor{tnames[i].data(), static_cast<uint32_t>(tnames[i].size()),
                               reinterpret_cast<const uint8_t*>("bfloat16"), 8, shapes[i].data(),
                               static_cast<uint32_t>(shapes[i].size()), rnd() % (1u << 30), root};
        }
        uint8_t ident[32];
        const int irc = pkv_content_identity(ts.data(), nt, f.data(), n, ident);
        check(irc == PKV_OK || irc == PKV_EDUPDIM, "content identity");
    }
    // size queries
    check(pkv_table_bytes(4) == 128 && pkv_table_bytes(6) == 0 && pkv_table_bytes(1ull << 57) == 0, "table bytes");
    for (int i = 0; i < 100; ++i) check(pkv_tree_work_bytes((rnd() % (1ull << 40)) & ~3ull, 1 + rnd() % 5000) > 0,
                                        "tree work bytes");
    // argument errors are returned before anything is launched
    pkv_table bad_table{nullptr, 1000};
    check(pkv_table_init(&bad_table, nullptr) == PKV_EINVAL, "init bad table");
    check(pkv_key_offsets(nullptr, 4, 16, nullptr, nullptr) == PKV_EINVAL, "key offsets null");
    check(pkv_derive_keys(nullptr, 0, nullptr, 4, nullptr, 0, nullptr, 0, nullptr, nullptr, nullptr) == PKV_EINVAL,
          "derive block 0");
    check(pkv_digest_batch(nullptr, 8, nullptr, nullptr, 3, nullptr, nullptr, nullptr) == PKV_EINVAL, "digest batch null");
    check(pkv_expand_digests(nullptr, 2, nullptr, 3, nullptr, nullptr, nullptr) == PKV_EINVAL, "expand null");
    check(pkv_tensor_roots_static(reinterpret_cast<const uint8_t*>(0x1000), 1ull << 28,
                                  reinterpret_cast<const int64_t*>(0x2000), reinterpret_cast<const int64_t*>(0x3000), 1,
                                  reinterpret_cast<uint8_t*>(0x4000), reinterpret_cast<int32_t*>(0x5000),
                                  nullptr) == PKV_EINVAL, "static roots too large");
    check(std::strlen(pkv_last_error()) > 0 && std::strlen(pkv_version()) > 0, "error text");
    return bad ? 1 : 0;
}
