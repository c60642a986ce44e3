// k_tree.hip -- content identities on gfx950: Merkle roots of tensors' bytes (section 5.3: an
// adapter is bound by an identity of its contents; section 6.5: what computing it costs).
//
// Tensor t occupies [tensor_off[t], tensor_off[t] + tensor_len[t]) of the data (4-byte aligned start).
// Tree of one tensor: leaves of 1024 bytes, leaf = SHA-256(0x00 | bytes); a node is
// SHA-256(0x01 | up to 16 consecutive child digests); the first level with a single digest holds
// the root (an empty tensor has one empty leaf).  All tensors are hashed together: level 0 has one
// lane per leaf of every tensor, each further level one lane per node.  Per level, a
// one-workgroup scan turns the tensors' node counts into offsets (CSR); a tensor whose tree is
// already a single digest carries it up unchanged.
//
// Work area (see tree_layout): the CSR of every level, then the digests of every level.
#include "pkv_internal.h"

namespace pkv {
namespace {

using dev::bswap;
using dev::compress;
using dev::init_state;

constexpr uint32_t kLeafBytes = 1024;
constexpr uint32_t kFanIn = 16;
constexpr int kCsrThreads = 1024;

// Big-endian data word k of a message of len bytes at p4 (4-byte aligned; the dword holding its
// last byte is readable), with the FIPS 180-4 padding byte 0x80 at byte len and zeros after.
__device__ __forceinline__ uint32_t data_word(const uint32_t* p4, uint32_t len, int64_t k) {
    if (k < 0) return 0u;
    if (len == 0) return k == 0 ? 0x80000000u : 0u;
    const int64_t last = (static_cast<int64_t>(len) - 1) >> 2;
    const uint32_t be = bswap(p4[k < last ? k : last]);
    const int64_t r = static_cast<int64_t>(len) - 4 * k;             // data bytes in this word
    const uint32_t keep = r >= 4 ? 0xFFFFFFFFu : (r <= 0 ? 0u : (0xFFFFFFFFu << (8 * (4 - r))));
    const uint32_t pad = (r >= 0 && r < 4) ? (0x80u << (8 * (3 - r))) : 0u;
    return (be & keep) | pad;
}

// SHA-256(prefix | data[0 .. len)): message word q takes the last byte of data word q - 1 (the
// prefix for q = 0) and the first three of data word q.
__device__ __forceinline__ void hash_prefixed(uint32_t prefix, const uint32_t* p4, uint32_t len, uint32_t s[8]) {
    const uint64_t msg = 1ull + len;
    const uint64_t n_blocks = (msg + 9 + 63) / 64;
    init_state(s);
    uint32_t carry = prefix;                                          // previous data word (low byte used)
    for (uint64_t c = 0; c < n_blocks; ++c) {
        uint32_t w[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const uint32_t cur = data_word(p4, len, static_cast<int64_t>(16 * c + q));
            w[q] = __builtin_amdgcn_alignbit(carry, cur, 8);
            carry = cur;
        }
        if (c + 1 == n_blocks) {
            w[14] = static_cast<uint32_t>((msg * 8) >> 32);
            w[15] = static_cast<uint32_t>(msg * 8);
        }
        compress(s, w);
    }
}

__device__ __forceinline__ void store_digest(uint8_t* d, uint64_t i, const uint32_t s[8]) {
    uint4* o = reinterpret_cast<uint4*>(d + 32 * i);
    o[0] = make_uint4(bswap(s[0]), bswap(s[1]), bswap(s[2]), bswap(s[3]));
    o[1] = make_uint4(bswap(s[4]), bswap(s[5]), bswap(s[6]), bswap(s[7]));
}

// Largest t in [0, n) with csr[t] <= i (csr non-decreasing, csr[0] = 0).
__device__ __forceinline__ uint32_t owner(const int64_t* csr, uint32_t n, int64_t i) {
    uint32_t lo = 0, hi = n;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (csr[mid] <= i) lo = mid; else hi = mid;
    }
    return lo;
}

// One workgroup: csr[t] = sum of count(t') over t' < t.  Level 0: count = leaves of tensor t
// (its offsets are validated: a bad tensor counts one leaf and reports PKV_ELAYOUT); level > 0:
// count = ceil(nodes of the level below / 16).
__global__ __launch_bounds__(kCsrThreads) void k_tree_csr(const int64_t* tensor_off, const int64_t* tensor_len,
                                                          uint64_t n_bytes, uint32_t n, const int64_t* below,
                                                          int64_t* csr, int32_t* status) {
    __shared__ int64_t wave_sum[kCsrThreads / 64];
    __shared__ int64_t carry;
    const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) { carry = 0; csr[0] = 0; }
    __syncthreads();
    for (uint32_t base = 0; base < n; base += kCsrThreads) {
        const uint32_t t = base + tid;
        int64_t cnt = 0;
        if (t < n) {
            if (below == nullptr) {
                const int64_t a = tensor_off[t], l = tensor_len[t];
                const bool ok = a >= 0 && l >= 0 && static_cast<uint64_t>(a) <= n_bytes &&
                                static_cast<uint64_t>(l) <= n_bytes - static_cast<uint64_t>(a) && (a & 3) == 0;
                if (!ok) dev::report(status, PKV_ELAYOUT);
                const int64_t len = ok ? l : 0;
                cnt = len == 0 ? 1 : (len + kLeafBytes - 1) / kLeafBytes;
            } else {
                cnt = (below[t + 1] - below[t] + kFanIn - 1) / kFanIn;
            }
        }
        int64_t incl = cnt;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int64_t y = __shfl_up(incl, d, 64);
            if (lane >= static_cast<uint32_t>(d)) incl += y;
        }
        if (lane == 63) wave_sum[wave] = incl;
        __syncthreads();
        int64_t wave_base = 0, total = 0;
        for (uint32_t q = 0; q < kCsrThreads / 64; ++q) {
            if (q < wave) wave_base += wave_sum[q];
            total += wave_sum[q];
        }
        if (t < n) csr[t + 1] = carry + wave_base + incl;
        __syncthreads();
        if (tid == 0) carry += total;
        __syncthreads();
    }
}

// Level 0: one lane per leaf of every tensor.
__global__ __launch_bounds__(64) void k_tree_leaves(const uint8_t* data, uint64_t n_bytes, const int64_t* tensor_off,
                                                    const int64_t* tensor_len, uint32_t n, const int64_t* csr,
                                                    uint8_t* out) {
    const int64_t i = blockIdx.x * 64ll + threadIdx.x;
    if (i >= csr[n]) return;
    const uint32_t t = owner(csr, n, i);
    const int64_t a = tensor_off[t], l = tensor_len[t];
    if (a < 0 || l < 0 || static_cast<uint64_t>(a) > n_bytes || static_cast<uint64_t>(l) > n_bytes - a || (a & 3) != 0)
        return;                                                       // reported by k_tree_csr
    const int64_t b = a + l;
    const int64_t j = i - csr[t];
    const int64_t start = a + j * kLeafBytes;
    const int64_t rem = b - start;
    const uint32_t len = rem <= 0 ? 0u : (rem < kLeafBytes ? static_cast<uint32_t>(rem) : kLeafBytes);
    uint32_t s[8];
    hash_prefixed(0x00u, reinterpret_cast<const uint32_t*>(data + start), len, s);
    store_digest(out, i, s);
}

// Level l > 0: one lane per node; children are the level below's digests of the same tensor.
__global__ __launch_bounds__(64) void k_tree_nodes(uint32_t n, const int64_t* csr_below, const int64_t* csr,
                                                   const uint8_t* below, uint8_t* out) {
    const int64_t i = blockIdx.x * 64ll + threadIdx.x;
    if (i >= csr[n]) return;
    const uint32_t t = owner(csr, n, i);
    const int64_t j = i - csr[t];
    const int64_t c0 = csr_below[t] + kFanIn * j;
    const int64_t end = csr_below[t + 1];
    const int64_t c1 = c0 + kFanIn < end ? c0 + kFanIn : end;
    if (end - csr_below[t] == 1) {                                    // already the root: carried up
        const uint4* src = reinterpret_cast<const uint4*>(below + 32 * c0);
        uint4* dst = reinterpret_cast<uint4*>(out + 32 * i);
        dst[0] = src[0];
        dst[1] = src[1];
        return;
    }
    uint32_t s[8];
    hash_prefixed(0x01u, reinterpret_cast<const uint32_t*>(below + 32 * c0), static_cast<uint32_t>(32 * (c1 - c0)), s);
    store_digest(out, i, s);
}

__global__ __launch_bounds__(256) void k_tree_roots(uint32_t n, const int64_t* csr, const uint8_t* top, uint8_t* roots) {
    const uint32_t t = blockIdx.x * 256 + threadIdx.x;
    if (t >= n) return;
    const uint4* src = reinterpret_cast<const uint4*>(top + 32 * csr[t]);
    uint4* dst = reinterpret_cast<uint4*>(roots + 32 * static_cast<uint64_t>(t));
    dst[0] = src[0];
    dst[1] = src[1];
}

}  // namespace

// Levels and work-area layout for n_bytes of data in n tensors (host and device agree on it).
TreeLayout tree_layout(uint64_t n_bytes, uint32_t n) {
    TreeLayout L{};
    uint64_t leaves_max = n_bytes / kLeafBytes + 1;                   // leaves of the largest tensor
    L.levels = 1;
    for (uint64_t c = leaves_max; c > 1; c = (c + kFanIn - 1) / kFanIn) ++L.levels;
    uint64_t bound = (n_bytes + kLeafBytes - 1) / kLeafBytes + n;     // leaves of all tensors
    uint64_t off = static_cast<uint64_t>(L.levels) * (n + 1ull) * 8;  // CSR arrays first
    off = (off + 255) & ~255ull;
    for (uint32_t l = 0; l < L.levels; ++l) {
        L.bound[l] = bound;
        L.digest_off[l] = off;
        off += bound * 32;
        bound = (bound + kFanIn - 1) / kFanIn + n;
    }
    L.bytes = off;
    return L;
}

int launch_tensor_roots(const uint8_t* data, uint64_t n_bytes, const int64_t* tensor_off, const int64_t* tensor_len,
                        uint32_t n, uint8_t* work, uint8_t* roots, int32_t* status, hipStream_t s) {
    if (n == 0) return PKV_OK;
    const TreeLayout L = tree_layout(n_bytes, n);
    int64_t* csr = reinterpret_cast<int64_t*>(work);
    auto csr_of = [&](uint32_t l) { return csr + static_cast<uint64_t>(l) * (n + 1ull); };
    hipLaunchKernelGGL(k_tree_csr, dim3(1), dim3(kCsrThreads), 0, s, tensor_off, tensor_len, n_bytes, n,
                       static_cast<const int64_t*>(nullptr), csr_of(0), status);
    hipLaunchKernelGGL(k_tree_leaves, dim3(static_cast<unsigned>((L.bound[0] + 63) / 64)), dim3(64), 0, s, data,
                       n_bytes, tensor_off, tensor_len, n, csr_of(0), work + L.digest_off[0]);
    for (uint32_t l = 1; l < L.levels; ++l) {
        hipLaunchKernelGGL(k_tree_csr, dim3(1), dim3(kCsrThreads), 0, s, tensor_off, tensor_len, n_bytes, n,
                           csr_of(l - 1), csr_of(l), status);
        hipLaunchKernelGGL(k_tree_nodes, dim3(static_cast<unsigned>((L.bound[l] + 63) / 64)), dim3(64), 0, s, n,
                           csr_of(l - 1), csr_of(l), work + L.digest_off[l - 1], work + L.digest_off[l]);
    }
    hipLaunchKernelGGL(k_tree_roots, dim3((n + 255) / 256), dim3(256), 0, s, n, csr_of(L.levels - 1),
                       work + L.digest_off[L.levels - 1], roots);
    return check_launch("pkv_tensor_roots");
}

}  // namespace pkv
