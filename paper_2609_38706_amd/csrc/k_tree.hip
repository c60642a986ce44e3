// k_tree.hip -- content identities on gfx950: Merkle roots of tensors' bytes (section 5.3: an
// adapter is bound by an identity of its contents; section 6.5: what computing it costs).
//
// Tensor t occupies [tensor_off[t], tensor_off[t] + tensor_len[t]) of the data (4-byte aligned start).
// Tree of one tensor: leaves of 1024 bytes, leaf = SHA-256(0x00 | bytes); a node is
// SHA-256(0x01 | up to 16 consecutive child digests); the first level with a single digest holds
// the root (an empty tensor has one empty leaf).  All tensors are hashed together: level 0 has one
// lane per leaf of every tensor, each further level one lane per node.  One workgroup first
// turns the tensors' node counts at every level into offsets (CSR); a tensor whose tree is
// already a single digest carries it up unchanged.
//
// Data that starts 16-byte aligned and is a whole number of 16-byte units (every full leaf of an
// aligned tensor; every node, since the work area is 256-byte aligned) is read with 16-byte loads,
// the next block while the current one compresses; other leaves take the byte-exact path.
//
// Work area (see tree_layout): the CSR of every level, then the digests of every level.
#include <mutex>

#include "pkv_internal.h"

// Work area of pkv_tensor_roots_static: one copy per device, held until the process ends.  Host code
// never passes this name to a kernel: it stands for a host-side shadow, not the device address;
// static_tree_work() resolves the address per device.
static __device__ __align__(256) uint8_t scratch[PKV_STATIC_TREE_WORK_BYTES];

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

__device__ __forceinline__ void load_units(const uint4* p, uint32_t n16, uint32_t u0, uint4 v[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t u = u0 + i;
        v[i] = p[u < n16 ? u : n16 - 1];                              // n16 > 0: clamped to the data
    }
}

// SHA-256(prefix | data[0 .. 16 n16)) for 16-byte-aligned data.  The stream of big-endian data words
// is followed by the padding word 0x80000000 and zeros; message word q takes the last byte of stream
// word q - 1 (the prefix for q = 0) and the first three of stream word q.  Blocks made only of data
// words skip the padding selects; at most two blocks follow them (the rest of the data, the padding,
// the length), and every data unit they hold is already loaded when the loop over full blocks ends.
__device__ __forceinline__ void hash_prefixed16(uint32_t prefix, const uint4* p, uint32_t n16, uint32_t s[8]) {
    const uint64_t msg = 1ull + 16ull * n16;
    const uint32_t n_full = n16 / 4;
    const uint32_t n_blocks = static_cast<uint32_t>((msg + 9 + 63) / 64);
    init_state(s);
    uint32_t carry = prefix;
    uint4 cur[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) cur[i] = make_uint4(0u, 0u, 0u, 0u);
    if (n16 > 0) load_units(p, n16, 0, cur);
    for (uint32_t c = 0; c < n_full; ++c) {
        uint32_t w[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t raw[4] = {cur[i].x, cur[i].y, cur[i].z, cur[i].w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t be = bswap(raw[k]);
                w[4 * i + k] = __builtin_amdgcn_alignbit(carry, be, 8);
                carry = be;
            }
        }
        load_units(p, n16, 4 * (c + 1), cur);
        __builtin_amdgcn_sched_barrier(0);                            // the loads stay ahead of the rounds
        compress(s, w);
    }
    for (uint32_t c = n_full; c < n_blocks; ++c) {
        uint32_t w[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t u = 4 * c + i;
            const bool in = u < n16;
            const uint32_t raw[4] = {cur[i].x, cur[i].y, cur[i].z, cur[i].w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t pad = (k == 0 && u == n16) ? 0x80000000u : 0u;
                const uint32_t be = in ? bswap(raw[k]) : pad;
                w[4 * i + k] = __builtin_amdgcn_alignbit(carry, be, 8);
                carry = be;
            }
        }
        if (c + 1 == n_blocks) {
            w[14] = static_cast<uint32_t>((msg * 8) >> 32);
            w[15] = static_cast<uint32_t>(msg * 8);
        }
        compress(s, w);
    }
}

__device__ __forceinline__ bool aligned16(const void* p, uint64_t len) {
    return ((reinterpret_cast<uintptr_t>(p) | len) & 15) == 0;
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

constexpr uint32_t kStagedCsr = 1024;                                 // CSR entries staged in LDS (8 KB)

// Tensor owning item i of a level, or n when i lies past the level.  When the level's CSR fits, it
// is staged in LDS first, so the search reads LDS instead of making dependent global loads.  Every
// lane of the workgroup must call it (the staging ends in a barrier).
__device__ __forceinline__ uint32_t find_owner(const int64_t* csr, uint32_t n, int64_t i, int64_t* lcsr) {
    if (n + 1 <= kStagedCsr) {
        for (uint32_t k = threadIdx.x; k <= n; k += blockDim.x) lcsr[k] = csr[k];
        __syncthreads();
        return i >= lcsr[n] ? n : owner(lcsr, n, i);
    }
    return i >= csr[n] ? n : owner(csr, n, i);
}

// Digests reserved per tree level in the work area (tree_layout), passed to the kernels by value.
struct LevelBounds {
    uint64_t b[32];
};

// One workgroup: the CSR of every level, csr_l[t] = sum over t' < t of the nodes of tensor t' at
// level l.  Level 0 counts the leaves of each tensor (its start and length are validated: a bad
// tensor counts one leaf and reports PKV_ELAYOUT); level l + 1 counts ceil(level l / 16).  Tensors
// whose lengths add up to more than the data are PKV_ELAYOUT as well: the work area reserves, per
// level, room for the nodes of tensors that fit the data side by side (tree_layout), and a level
// whose node total exceeds its reservation is reported the same way.  The hashing kernels never
// index past a level's reservation, so such input yields unspecified roots but no access outside
// the work area.
__global__ __launch_bounds__(kCsrThreads) void k_tree_csr(const int64_t* tensor_off, const int64_t* tensor_len,
                                                          uint64_t n_bytes, uint32_t n, uint32_t levels,
                                                          LevelBounds bounds, int64_t* csr, int32_t* status) {
    __shared__ int64_t wave_sum[kCsrThreads / 64];
    __shared__ uint64_t wave_bytes[kCsrThreads / 64];
    __shared__ int64_t carry;
    __shared__ uint64_t byte_total;
    const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (uint32_t l = 0; l < levels; ++l) {
        int64_t* out = csr + static_cast<uint64_t>(l) * (n + 1ull);
        if (tid == 0) { carry = 0; byte_total = 0; out[0] = 0; }
        __syncthreads();
        for (uint32_t base = 0; base < n; base += kCsrThreads) {
            const uint32_t t = base + tid;
            int64_t cnt = 0;
            uint64_t bytes = 0;
            if (t < n) {
                const int64_t a = tensor_off[t], len = tensor_len[t];
                const bool ok = a >= 0 && len >= 0 && static_cast<uint64_t>(a) <= n_bytes &&
                                static_cast<uint64_t>(len) <= n_bytes - static_cast<uint64_t>(a) && (a & 3) == 0;
                if (!ok && l == 0) dev::report(status, PKV_ELAYOUT);
                bytes = ok ? static_cast<uint64_t>(len) : 0u;
                cnt = bytes == 0 ? 1 : static_cast<int64_t>((bytes + kLeafBytes - 1) / kLeafBytes);
                for (uint32_t k = 0; k < l; ++k) cnt = (cnt + kFanIn - 1) / kFanIn;
            }
            int64_t incl = cnt;
            uint64_t bsum = bytes;                            // each length <= n_bytes < 2^56: no overflow
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int64_t y = __shfl_up(incl, d, 64);
                if (lane >= static_cast<uint32_t>(d)) incl += y;
                bsum += __shfl_xor(bsum, d, 64);
            }
            if (lane == 63) wave_sum[wave] = incl;
            if (lane == 0) wave_bytes[wave] = bsum;
            __syncthreads();
            int64_t wave_base = 0, total = 0;
            uint64_t btotal = 0;
            for (uint32_t q = 0; q < kCsrThreads / 64; ++q) {
                if (q < wave) wave_base += wave_sum[q];
                total += wave_sum[q];
                btotal += wave_bytes[q];
            }
            if (t < n) out[t + 1] = carry + wave_base + incl;
            __syncthreads();
            if (tid == 0) {
                carry += total;
                byte_total += btotal;
            }
            __syncthreads();
        }
        if (tid == 0 && ((l == 0 && byte_total > n_bytes) || static_cast<uint64_t>(carry) > bounds.b[l]))
            dev::report(status, PKV_ELAYOUT);
    }
}

// Level 0: one lane per leaf of every tensor.
__global__ __launch_bounds__(64) void k_tree_leaves(const uint8_t* data, uint64_t n_bytes, const int64_t* tensor_off,
                                                    const int64_t* tensor_len, uint32_t n, const int64_t* csr,
                                                    uint64_t bound, uint8_t* out) {
    __shared__ int64_t lcsr[kStagedCsr];
    const int64_t i = blockIdx.x * 64ll + threadIdx.x;
    const uint32_t t = find_owner(csr, n, i, lcsr);
    if (t == n || static_cast<uint64_t>(i) >= bound) return;       // past the level's reservation
    const int64_t a = tensor_off[t], l = tensor_len[t];
    if (a < 0 || l < 0 || static_cast<uint64_t>(a) > n_bytes || static_cast<uint64_t>(l) > n_bytes - a || (a & 3) != 0)
        return;                                                       // reported by k_tree_csr
    const int64_t b = a + l;
    const int64_t j = i - csr[t];
    const int64_t start = a + j * kLeafBytes;
    const int64_t rem = b - start;
    const uint32_t len = rem <= 0 ? 0u : (rem < kLeafBytes ? static_cast<uint32_t>(rem) : kLeafBytes);
    uint32_t s[8];
    if (aligned16(data + start, len))
        hash_prefixed16(0x00u, reinterpret_cast<const uint4*>(data + start), len / 16, s);
    else
        hash_prefixed(0x00u, reinterpret_cast<const uint32_t*>(data + start), len, s);
    store_digest(out, i, s);
}

// Level l > 0: one lane per node; children are the level below's digests of the same tensor.
__global__ __launch_bounds__(64) void k_tree_nodes(uint32_t n, const int64_t* csr_below, const int64_t* csr,
                                                   const uint8_t* below, uint64_t bound_below, uint64_t bound,
                                                   uint8_t* out) {
    __shared__ int64_t lcsr[kStagedCsr];
    const int64_t i = blockIdx.x * 64ll + threadIdx.x;
    const uint32_t t = find_owner(csr, n, i, lcsr);
    if (t == n || static_cast<uint64_t>(i) >= bound) return;       // past the level's reservation
    const int64_t j = i - csr[t];
    const int64_t c0 = csr_below[t] + kFanIn * j;
    const int64_t end = csr_below[t + 1];
    const int64_t c1 = c0 + kFanIn < end ? c0 + kFanIn : end;
    if (c0 < 0 || c1 <= c0 || static_cast<uint64_t>(c1) > bound_below) return;   // children past the level below
    if (end - csr_below[t] == 1) {                                    // already the root: carried up
        const uint4* src = reinterpret_cast<const uint4*>(below + 32 * c0);
        uint4* dst = reinterpret_cast<uint4*>(out + 32 * i);
        dst[0] = src[0];
        dst[1] = src[1];
        return;
    }
    uint32_t s[8];                                                    // digests are 32-byte aligned
    hash_prefixed16(0x01u, reinterpret_cast<const uint4*>(below + 32 * c0), static_cast<uint32_t>(2 * (c1 - c0)), s);
    store_digest(out, i, s);
}

__global__ __launch_bounds__(256) void k_tree_roots(uint32_t n, const int64_t* csr, const uint8_t* top, uint64_t bound,
                                                    uint8_t* roots) {
    const uint32_t t = blockIdx.x * 256 + threadIdx.x;
    if (t >= n) return;
    uint4* dst = reinterpret_cast<uint4*>(roots + 32 * static_cast<uint64_t>(t));
    const int64_t at = csr[t];
    if (at < 0 || static_cast<uint64_t>(at) >= bound) {                // reported by k_tree_csr
        dst[0] = make_uint4(0u, 0u, 0u, 0u);
        dst[1] = make_uint4(0u, 0u, 0u, 0u);
        return;
    }
    const uint4* src = reinterpret_cast<const uint4*>(top + 32 * at);
    dst[0] = src[0];
    dst[1] = src[1];
}

}  // namespace

// Levels and work-area layout for n_bytes of data in n tensors (host and device agree on it).  The
// reservation of a level holds the nodes of any tensors whose lengths sum to at most n_bytes: level
// 0 has sum of max(1, ceil(len_t / 1024)) <= n_bytes / 1024 + n leaves, and a level of T nodes has
// at most T / 16 + n parents.
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

// Device address of `scratch` on the current device, looked up once per device (with that device
// current) and kept.
int static_tree_work(uint8_t** out) {
    static std::mutex mu;
    static void* addr[64] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return set_error(PKV_EHIP, "pkv_tensor_roots_static: hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= 64) return set_error(PKV_EINVAL, "pkv_tensor_roots_static: device %d out of range", dev);
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return set_error(PKV_EHIP, "pkv_tensor_roots_static: hipGetSymbolAddress: %s", hipGetErrorString(e));
        addr[dev] = p;
    }
    *out = static_cast<uint8_t*>(addr[dev]);
    return PKV_OK;
}

int launch_tensor_roots(const uint8_t* data, uint64_t n_bytes, const int64_t* tensor_off, const int64_t* tensor_len,
                        uint32_t n, uint8_t* work, uint8_t* roots, int32_t* status, hipStream_t s) {
    if (n == 0) return PKV_OK;
    const TreeLayout L = tree_layout(n_bytes, n);
    int64_t* csr = reinterpret_cast<int64_t*>(work);
    auto csr_of = [&](uint32_t l) { return csr + static_cast<uint64_t>(l) * (n + 1ull); };
    LevelBounds bounds{};
    for (uint32_t l = 0; l < L.levels; ++l) bounds.b[l] = L.bound[l];
    hipLaunchKernelGGL(k_tree_csr, dim3(1), dim3(kCsrThreads), 0, s, tensor_off, tensor_len, n_bytes, n, L.levels,
                       bounds, csr, status);
    hipLaunchKernelGGL(k_tree_leaves, dim3(static_cast<unsigned>((L.bound[0] + 63) / 64)), dim3(64), 0, s, data,
                       n_bytes, tensor_off, tensor_len, n, csr_of(0), L.bound[0], work + L.digest_off[0]);
    for (uint32_t l = 1; l < L.levels; ++l) {
        hipLaunchKernelGGL(k_tree_nodes, dim3(static_cast<unsigned>((L.bound[l] + 63) / 64)), dim3(64), 0, s, n,
                           csr_of(l - 1), csr_of(l), work + L.digest_off[l - 1], L.bound[l - 1], L.bound[l],
                           work + L.digest_off[l]);
    }
    hipLaunchKernelGGL(k_tree_roots, dim3((n + 255) / 256), dim3(256), 0, s, n, csr_of(L.levels - 1),
                       work + L.digest_off[L.levels - 1], L.bound[L.levels - 1], roots);
    return check_launch("pkv_tensor_roots");
}

}  // namespace pkv
