// k_derive.hip -- descriptor digests, key offsets and chained block keys on gfx950.
//
// Key chain (section 5.2, Eq. 3 with f = a chained block key):
//   key_i = H(key_{i-1} | d | LE32 tokens of block i),  key_0 = 0^16,  H = SHA-256[0:16].
// The message of one key is 32 + 4B bytes = 8 + B big-endian words:
//   words 0-3   key_{i-1} (the previous SHA-256 state words H0..H3 feed straight back in),
//   words 4-7   the descriptor digest,
//   words 8..   the byte-swapped int32 tokens of the block,
//   then FIPS 180-4 padding (0x80000000, zeros, 64-bit bit length).
// A chain is strictly serial, so one lane owns one request and a wavefront owns 64 requests;
// all work is 32-bit integer VALU (v_alignbit rotates, v_bitop3/v_bfi logic, v_add3 sums,
// v_perm byte swaps).
#include <atomic>

#include "pkv_internal.h"

namespace pkv {
namespace {

using dev::bswap;
using dev::compress;
using dev::init_state;

constexpr int kDeriveThreads = 64;   // one wavefront per workgroup: 64 independent chains

struct ChainArgs {
    const int32_t* tokens;
    uint64_t n_tokens;
    const int64_t* tok_off;
    uint32_t n_req;
    const uint8_t* digests;
    uint32_t block;
    const int64_t* key_off;
    uint64_t n_keys;
    uint8_t* keys;
    int32_t* status;
    // fused derive and lookup only (else null / 0): the index buckets, the bucket count - 1 and
    // the per-request hit lengths
    const uint4* table;
    uint64_t bucket_mask;
    int32_t* hits;
};

// Loads request r's bounds and checks them against the buffers; false = skip this request.
__device__ __forceinline__ bool chain_bounds(const ChainArgs& a, uint32_t r, int64_t& t0, int64_t& k0,
                                             int64_t& n) {
    t0 = a.tok_off[r];
    const int64_t t1 = a.tok_off[r + 1];
    k0 = a.key_off[r];
    const int64_t k1 = a.key_off[r + 1];
    const bool ok = t0 >= 0 && t1 >= t0 && static_cast<uint64_t>(t1) <= a.n_tokens && k0 >= 0 && k1 >= k0 &&
                    static_cast<uint64_t>(k1) <= a.n_keys && (k1 - k0) == (t1 - t0) / a.block;
    if (!ok) {
        dev::report(a.status, PKV_ELAYOUT);
        return false;
    }
    n = k1 - k0;
    return true;
}

__device__ __forceinline__ void load_digest(const ChainArgs& a, uint32_t r, uint32_t d[4]) {
    const uint4 v = reinterpret_cast<const uint4*>(a.digests)[r];
    d[0] = bswap(v.x); d[1] = bswap(v.y); d[2] = bswap(v.z); d[3] = bswap(v.w);
}

__device__ __forceinline__ void store_key(uint8_t* keys, int64_t idx, const uint32_t s[8]) {
    reinterpret_cast<uint4*>(keys)[idx] = make_uint4(bswap(s[0]), bswap(s[1]), bswap(s[2]), bswap(s[3]));
}

// ---- B = 16: two compressions per key; the next key's 16 tokens are prefetched -------------
__global__ __launch_bounds__(kDeriveThreads) void k_derive_b16(ChainArgs a) {
    const uint32_t r = blockIdx.x * kDeriveThreads + threadIdx.x;
    if (r >= a.n_req) return;
    int64_t t0, k0, n;
    if (!chain_bounds(a, r, t0, k0, n)) return;
    uint32_t dg[4], prev[4] = {0u, 0u, 0u, 0u};
    load_digest(a, r, dg);
    const int32_t* tp = a.tokens + t0;
    uint32_t nxt[16];
    if (n > 0) {
#pragma unroll
        for (int q = 0; q < 16; ++q) nxt[q] = static_cast<uint32_t>(tp[q]);
    }
    for (int64_t i = 0; i < n; ++i) {
        uint32_t cur[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) cur[q] = nxt[q];
        if (i + 1 < n) {
            const int32_t* np = tp + (i + 1) * 16;
#pragma unroll
            for (int q = 0; q < 16; ++q) nxt[q] = static_cast<uint32_t>(np[q]);
        }
        uint32_t s[8], w[16];
        init_state(s);
#pragma unroll
        for (int q = 0; q < 4; ++q) { w[q] = prev[q]; w[4 + q] = dg[q]; }
#pragma unroll
        for (int q = 0; q < 8; ++q) w[8 + q] = bswap(cur[q]);
        compress(s, w);
#pragma unroll
        for (int q = 0; q < 8; ++q) w[q] = bswap(cur[8 + q]);
        w[8] = 0x80000000u;
#pragma unroll
        for (int q = 9; q < 15; ++q) w[q] = 0u;
        w[15] = (32u + 4u * 16u) * 8u;
        compress(s, w);
        store_key(a.keys, k0 + i, s);
#pragma unroll
        for (int q = 0; q < 4; ++q) prev[q] = s[q];
    }
}

// ---- consumer / helper split (used while chains are scarce) -----------------------------------
// A chain's rounds are strictly serial, but much of each key's instruction stream is not on that
// serial path.  Two wavefronts share the same chains:
//   consumer: only the SHA-256 rounds of every key, reading K_t + W_t from LDS;
//   helper:   during the first three phases of key i, compression 1's schedule W16..W63 (it
//             depends on key i-1), one phase ahead of the consumer; during the long last phase,
//             every token-only part of key i+1 (token loads two keys ahead, byte swaps, the whole
//             schedule of the token-only compressions) into a double buffer.
// Per key there are four phases separated by workgroup barriers: phases 0-2 each hold 16 rounds
// of compression 1, phase 3 holds its last 16 rounds and the token-only compressions, whose K + W
// words the consumer already holds in registers.  The kernels below use this split with their
// rounds on lane pairs (B = 16: k_derive_b16_pp; B = 16m: k_derive_m16_pp) or one lane per chain
// (B = 16m: k_derive_m16_pc).
constexpr int kPcThreads = 128;

__device__ __forceinline__ void put4(uint4* p, const uint32_t* v) { *p = make_uint4(v[0], v[1], v[2], v[3]); }
__device__ __forceinline__ void get4(const uint4* p, uint32_t* v) {
    const uint4 x = *p;
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
}

// 16 consecutive rounds; kw[j] = K_{t0+j} + W_{t0+j}.  16 is a multiple of 8, so the state array
// keeps its naming across calls.
__device__ __forceinline__ void rounds16(uint32_t s[8], const uint32_t* kw) {
    uint32_t a = s[0], b = s[1], c = s[2], d = s[3], e = s[4], f = s[5], g = s[6], h = s[7];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const uint32_t t1 = h + dev::bsig1(e) + dev::choose(e, f, g) + kw[j];
        const uint32_t t2 = dev::bsig0(a) + dev::majority(a, b, c);
        h = g; g = f; f = e; e = d + t1;
        d = c; c = b; b = a; a = t1 + t2;
    }
    s[0] = a; s[1] = b; s[2] = c; s[3] = d; s[4] = e; s[5] = f; s[6] = g; s[7] = h;
}

// 16 schedule steps t = T0 .. T0+15 (T0 >= 16) on the rolling window w; kw receives K_t + W_t.
template <int T0>
__device__ __forceinline__ void schedule16(uint32_t w[16], uint32_t kw[16]) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int t = T0 + j;
        const uint32_t x = dev::ssig1(w[(t - 2) & 15]) + w[(t - 7) & 15] + dev::ssig0(w[(t - 15) & 15]) + w[t & 15];
        w[t & 15] = x;
        kw[j] = x + kRoundK[t];
    }
}

template <unsigned N>
__device__ __forceinline__ void lds_put16(uint4 (*dst)[N], uint32_t lane, const uint32_t kw[16]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) put4(&dst[q][lane], kw + 4 * q);
}
__device__ __forceinline__ void lds_get16(const uint4 (*src)[64], uint32_t lane, uint32_t* kw) {
#pragma unroll
    for (int q = 0; q < 4; ++q) get4(&src[q][lane], kw + 4 * q);
}

__device__ __forceinline__ int64_t wave_max(int64_t v) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t o = __shfl_xor(v, d, 64);
        v = v > o ? v : o;
    }
    return v;
}

// A value equal on every lane, moved to scalar registers (a loop bounded by it then runs as a
// scalar loop instead of an exec-mask loop).
__device__ __forceinline__ int64_t uniform64(int64_t v) {
    const uint64_t u = static_cast<uint64_t>(v);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// ---- B = 16, each chain on a lane pair (used while chains are very scarce) ---------------------
// Within one SHA-256 round the e-half (Sigma1, Ch, h + K_t + W_t) and the a-half (Sigma0, Maj) are
// independent until the final sums.  The consumer wavefront gives each chain two lanes, lane i and
// lane i + 8 of a 16-lane row: the first (the e lane, lanes 0..7 of each row) holds e, f, g, h, the
// second (the a lane, lanes 8..15; `odd` below, as it also computes the odd schedule words) holds
// a, b, c, d.  Both lanes run one instruction stream:
//   * three rotates with per-lane amounts and a 3-input XOR give Sigma1 / Sigma0;
//   * Maj(a, b, c) = Ch(~(a ^ b), b, c), so one select operand (x0 on the e lane, ~(x0 ^ x1) on the
//     a lane) and one Ch give Ch / Maj;
//   * Y = Sigma + Ch/Maj + Q, where Q = h + K_t + W_t on the e lane and 0 on the a lane, so Y = T1
//     on the e lane and Sigma0 + Maj on the a lane;
//   * two adds that read the partner lane (DPP row_ror:8 swaps the two halves of a row) and write
//     only one half of the row (DPP bank mask: lanes 0..7 or 8..15): e' = d + T1 on the e lane and
//     a' = T1 + Sigma0 + Maj on the a lane;
//   * Q of the next round, h' + K + W, by one more add written to the e lanes only (the a lanes'
//     Q stays zero).
// That is 10 instructions per round per wavefront instead of 14, which shortens the serial chain
// by 29% at 32 chains per wavefront.  The rounds are written as fixed instruction blocks: the e
// lane's add and the Q add sit between the producer of Y and the a lane's DPP read of it, which
// covers the two wait states a DPP read of a just-written register needs.  The helper wavefront
// splits each chain's message schedule the same way (even words on the e lane, odd words on the a
// lane), so it keeps ahead of the faster consumer; the token-only work of the next key is split the
// same way.
constexpr uint32_t kPpChains = 32;

// K + W words the consumer reads are split by parity: [p][r][chain] holds the words
// t = t0 + 8r + p + 2j (j = 0..3) for the lane of parity p (0: e lane, 1: a lane), so each lane
// reads four words of its own parity with one 16-byte load, and a round takes its Q word from its
// own lane or, for odd t, from the partner lane by DPP.
struct PpShared {
    uint4 kw2[2][2][8][kPpChains];    // K_t + W_t of compression 2 (t0 = 0), two keys; word 0 + h0
    uint4 w1tok[2][2][kPpChains];     // W8..W15 of compression 1, two keys (helper only)
    uint4 kw1tok[2][2][kPpChains];    // K_t + W_t, t = 8..15 of compression 1 (t0 = 8), two keys
    uint4 kw1hi[2][6][kPpChains];     // K_t + W_t, t = 16..63 of compression 1 (t0 = 16), current key
    uint4 prev[2][kPpChains];         // [1]: previous key words (a lanes); [0]: the e lanes' unused copy
};

struct PairLane {
    uint32_t m, nm, r1, r2, r3;       // all-ones on the a lane; its rotate amounts
};

// The lane's chain (0..31) and half of its pair: lanes i and i + 8 of each 16-lane row (lanes
// 0..7 of each row are e lanes).  The partner is read with DPP row_ror:8, and a DPP bank mask
// writes one half of a row.
__device__ __forceinline__ uint32_t pair_chain(uint32_t lane) { return ((lane >> 4) << 3) | (lane & 7u); }
__device__ __forceinline__ bool pair_is_a(uint32_t lane) { return (lane & 8u) != 0; }

// One paired round with the operand roles (x0, x1, x2, x3): the new x0 is written into x3's
// register and Q of the next round is formed from x2 (next round's x3) and KWN.  Bit tables of
// v_bitop3 index the operands as (S0, S1, S2) = (0xF0, 0xCC, 0xAA): 0x96 = 3-input XOR,
// 0xCA = S0 ? S1 : S2, 0xD2 = S2 ? ~(S0 ^ S1) : S0.  Four rounds in a row rotate the roles once
// around, so afterwards the state registers hold (x0, x1, x2, x3) in the same roles again.
#define PKV_ROUND_HEAD(X0, X1, X2)                                                                 \
    "v_alignbit_b32 %[t0], %[" #X0 "], %[" #X0 "], %[r1]\n"                                       \
    "v_alignbit_b32 %[t1], %[" #X0 "], %[" #X0 "], %[r2]\n"                                       \
    "v_alignbit_b32 %[t2], %[" #X0 "], %[" #X0 "], %[r3]\n"                                       \
    "v_bitop3_b32 %[t0], %[t0], %[t1], %[t2] bitop3:0x96\n"                                       \
    "v_bitop3_b32 %[t1], %[" #X0 "], %[" #X1 "], %[m] bitop3:0xd2\n"                              \
    "v_bitop3_b32 %[t1], %[t1], %[" #X1 "], %[" #X2 "] bitop3:0xca\n"                             \
    "v_add3_u32 %[t0], %[t0], %[t1], %[q]\n"
// On the e lane x3 is h, which only Q used, and e' = d + T1 overwrites it; on the a lane x3 is
// d, which the partner has read by then, and a' = T1 + Sigma0 + Maj overwrites it.  The e lane's
// add and the Q add sit between Y and the a lane's DPP read of it (two wait states).
#define PKV_PAIR_ROUND(X0, X1, X2, X3, KWN)                                                          \
    PKV_ROUND_HEAD(X0, X1, X2)                                                                    \
    "v_add_u32_dpp %[" #X3 "], %[" #X3 "], %[t0] row_ror:8 row_mask:0xf bank_mask:0x3\n"          \
    "v_add_u32_dpp %[q], %[" #X2 "], %[" #KWN "] quad_perm:[0,1,2,3] row_mask:0xf bank_mask:0x3\n" \
    "v_add_u32_dpp %[" #X3 "], %[t0], %[t0] row_ror:8 row_mask:0xf bank_mask:0xc\n"
// gfx950 fetches 8-byte instructions (VOP3, DPP) that are not 8-byte aligned at about one cycle
// more each: a run of the 10-instruction round placed 4 bytes off takes 50 cycles instead of 40.
// The compiler puts 4-byte instructions (s_nop, VOP2) between asm statements, so each block of
// rounds starts by padding itself back to an 8-byte boundary (the assembler pads with s_nop).
#define PKV_ALIGN8 ".p2align 3\n"

// 16 paired rounds as one asm statement, for K + W words that are all in registers already (the
// compiler's separator and the alignment padding then come once per 16 rounds instead of once
// per 4).  kw[j] = K + W of round t0 + j, `after` = K + W of round t0 + 16.
#define PKV_PAIR_ROUNDS4(K1, K2, K3, K4)                                                            \
    PKV_PAIR_ROUND(a, b, c, d, K1) PKV_PAIR_ROUND(d, a, b, c, K2) PKV_PAIR_ROUND(c, d, a, b, K3)      \
    PKV_PAIR_ROUND(b, c, d, a, K4)
__device__ __forceinline__ void pair_rounds16_regs(uint32_t x[4], uint32_t& q, const PairLane& pl, const uint32_t* kw,
                                                   uint32_t after) {
    uint32_t t0, t1, t2;
    asm volatile(PKV_ALIGN8 PKV_PAIR_ROUNDS4(k1, k2, k3, k4) PKV_PAIR_ROUNDS4(k5, k6, k7, k8)
                     PKV_PAIR_ROUNDS4(k9, k10, k11, k12) PKV_PAIR_ROUNDS4(k13, k14, k15, k16)
                 : [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [q] "+v"(q), [a] "+v"(x[0]), [b] "+v"(x[1]),
                   [c] "+v"(x[2]), [d] "+v"(x[3])
                 : [m] "v"(pl.m), [r1] "v"(pl.r1), [r2] "v"(pl.r2), [r3] "v"(pl.r3), [k1] "v"(kw[1]),
                   [k2] "v"(kw[2]), [k3] "v"(kw[3]), [k4] "v"(kw[4]), [k5] "v"(kw[5]), [k6] "v"(kw[6]),
                   [k7] "v"(kw[7]), [k8] "v"(kw[8]), [k9] "v"(kw[9]), [k10] "v"(kw[10]), [k11] "v"(kw[11]),
                   [k12] "v"(kw[12]), [k13] "v"(kw[13]), [k14] "v"(kw[14]), [k15] "v"(kw[15]), [k16] "v"(after));
}
#undef PKV_PAIR_ROUNDS4
#undef PKV_ALIGN8
#undef PKV_PAIR_ROUND
#undef PKV_ROUND_HEAD

// v of the pair's other lane (DPP row_ror:8).
__device__ __forceinline__ uint32_t lane_swap(uint32_t v) {
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x128, 0xF, 0xF, false));
}

// ---- k_derive_b16_pp's consumer: rounds with K + W split over the lane pair ------------------
// The e lane forms Q = h + K_t + W_t for the next round; K + W of even t sits in its own register,
// of odd t in the same register of its partner (the a lane), read by DPP row_ror:8.  So each lane
// holds half of a key's K + W words.  Every write of Q is masked to the e lanes (the a lanes' Q
// stays zero).  A block of rounds may start from read-only input registers (the chaining value)
// and write its first four new state words into fresh registers, which saves copying the input.
// Operand roles and instruction forms are those of the rounds above (PKV_ROUND_HEAD).
#define PKV_S_HEAD(X0, X1, X2)                                                                    \
    "v_alignbit_b32 %[t0], %[" #X0 "], %[" #X0 "], %[r1]\n"                                       \
    "v_alignbit_b32 %[t1], %[" #X0 "], %[" #X0 "], %[r2]\n"                                       \
    "v_alignbit_b32 %[t2], %[" #X0 "], %[" #X0 "], %[r3]\n"                                       \
    "v_bitop3_b32 %[t0], %[t0], %[t1], %[t2] bitop3:0x96\n"                                       \
    "v_bitop3_b32 %[t1], %[" #X0 "], %[" #X1 "], %[m] bitop3:0xd2\n"                              \
    "v_bitop3_b32 %[t1], %[t1], %[" #X1 "], %[" #X2 "] bitop3:0xca\n"                             \
    "v_add3_u32 %[t0], %[t0], %[t1], %[q]\n"
// next Q from the lane's own word / the partner's word / none (last round of a key)
#define PKV_QO(X2, K) "v_add_u32_dpp %[q], %[" #X2 "], %[" #K "] quad_perm:[0,1,2,3] row_mask:0xf bank_mask:0x3\n"
#define PKV_QP(X2, K) "v_add_u32_dpp %[q], %[" #K "], %[" #X2 "] row_ror:8 row_mask:0xf bank_mask:0x3\n"
#define PKV_QN(X2, K) "s_nop 0\n"
// one round: the new x0 goes to D (X3's register in place, or a fresh one)
#define PKV_SR(X0, X1, X2, X3, D, QF, K)                                                          \
    PKV_S_HEAD(X0, X1, X2)                                                                        \
    "v_add_u32_dpp %[" #D "], %[" #X3 "], %[t0] row_ror:8 row_mask:0xf bank_mask:0x3\n"           \
    QF(X2, K)                                                                                     \
    "v_add_u32_dpp %[" #D "], %[t0], %[t0] row_ror:8 row_mask:0xf bank_mask:0xc\n"
// in place, by position in the four-round cycle of roles
#define PKV_R0(QF, K) PKV_SR(a, b, c, d, d, QF, K)
#define PKV_R1(QF, K) PKV_SR(d, a, b, c, c, QF, K)
#define PKV_R2(QF, K) PKV_SR(c, d, a, b, b, QF, K)
#define PKV_R3(QF, K) PKV_SR(b, c, d, a, a, QF, K)
// from inputs i0..i3 into fresh a..d; afterwards a..d hold the roles x0..x3
#define PKV_F0(QF, K) PKV_SR(i0, i1, i2, i3, d, QF, K)
#define PKV_F1(QF, K) PKV_SR(d, i0, i1, i2, c, QF, K)
#define PKV_F2(QF, K) PKV_SR(c, d, i0, i1, b, QF, K)
#define PKV_F3(QF, K) PKV_SR(b, c, d, i0, a, QF, K)
// four rounds t0 + 4s .. of a phase whose own words are W[2s], W[2s+1] (K + W of t0 + 4s + 1 +
// j: partner's W[2s], own W[2s+1], partner's W[2s+1], own W[2s+2] is the next block's)
#define PKV_PH4(KA, KB) PKV_R0(PKV_QO, KA) PKV_R1(PKV_QP, KA) PKV_R2(PKV_QO, KB) PKV_R3(PKV_QP, KB)
#define PKV_ALIGN ".p2align 3\n"
#define PKV_S_IN [m] "v"(pl.m), [r1] "v"(pl.r1), [r2] "v"(pl.r2), [r3] "v"(pl.r3)
#define PKV_S_INOUT(X)                                                                            \
    [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [q] "+v"(q), [a] "+v"(X[0]), [b] "+v"(X[1]), \
        [c] "+v"(X[2]), [d] "+v"(X[3])
#define PKV_S_FRESH(X)                                                                            \
    [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [q] "+v"(q), [a] "=&v"(X[0]), [b] "=&v"(X[1]), \
        [c] "=&v"(X[2]), [d] "=&v"(X[3])

// After a block of n rounds in place the roles have turned n times: x0 moves to the register of
// x3, and so on.
__device__ __forceinline__ void roles_turn1(uint32_t x[4]) {
    const uint32_t t = x[3];
    x[3] = x[2]; x[2] = x[1]; x[1] = x[0]; x[0] = t;
}
__device__ __forceinline__ void roles_turn3(uint32_t x[4]) {
    const uint32_t t = x[0];
    x[0] = x[1]; x[1] = x[2]; x[2] = x[3]; x[3] = t;
}

// Q of round 0 (h0 + K_0 + W_0, into the e lanes of q) and K + W of rounds 1..3 from the partner's
// key words v: four DPP adds.  v was written well before (a workgroup barrier lies between), and
// s_nop 1 covers the two wait states a DPP read of a freshly written VGPR would need anyway.
__device__ __forceinline__ void swap_q_add3(uint32_t& q, uint32_t out[4], const uint32_t v[4], const uint32_t k[4]) {
    asm volatile("s_nop 1\n"
                 "v_add_u32_dpp %[q], %[v0], %[k0] row_ror:8 row_mask:0xf bank_mask:0x3\n"
                 "v_add_u32_dpp %[o1], %[v1], %[k1] row_ror:8 row_mask:0xf bank_mask:0xf\n"
                 "v_add_u32_dpp %[o2], %[v2], %[k2] row_ror:8 row_mask:0xf bank_mask:0xf\n"
                 "v_add_u32_dpp %[o3], %[v3], %[k3] row_ror:8 row_mask:0xf bank_mask:0xf"
                 : [q] "+v"(q), [o1] "=&v"(out[1]), [o2] "=&v"(out[2]), [o3] "=&v"(out[3])
                 : [v0] "v"(v[0]), [v1] "v"(v[1]), [v2] "v"(v[2]), [v3] "v"(v[3]), [k0] "v"(k[0]), [k1] "v"(k[1]),
                   [k2] "v"(k[2]), [k3] "v"(k[3]));
}

// Compression 1, rounds 0..6 from the initial value iv (K + W of rounds 1..3: kw[1..3], 4..7: dg).
__device__ __forceinline__ void pair_c1_r0_6(uint32_t x[4], uint32_t& q, const PairLane& pl, const uint32_t iv[4],
                                            const uint32_t kw[4], const uint32_t dg[4]) {
    uint32_t t0, t1, t2;
    asm volatile(PKV_ALIGN PKV_F0(PKV_QO, k1) PKV_F1(PKV_QO, k2) PKV_F2(PKV_QO, k3) PKV_F3(PKV_QO, k4)
                     PKV_R0(PKV_QO, k5) PKV_R1(PKV_QO, k6) PKV_R2(PKV_QO, k7)
                 : PKV_S_FRESH(x)
                 : PKV_S_IN, [i0] "v"(iv[0]), [i1] "v"(iv[1]), [i2] "v"(iv[2]), [i3] "v"(iv[3]), [k1] "v"(kw[1]),
                   [k2] "v"(kw[2]), [k3] "v"(kw[3]), [k4] "v"(dg[0]), [k5] "v"(dg[1]), [k6] "v"(dg[2]),
                   [k7] "v"(dg[3]));
    roles_turn3(x);
}

// Compression 1, rounds 7..11 (K + W of rounds 8..12 from the token words r: t = 8 + odd + 2j).
__device__ __forceinline__ void pair_c1_r7_11(uint32_t x[4], uint32_t& q, const PairLane& pl, const uint32_t r[4]) {
    uint32_t t0, t1, t2;
    asm volatile(PKV_ALIGN PKV_R0(PKV_QO, w0) PKV_R1(PKV_QP, w0) PKV_R2(PKV_QO, w1) PKV_R3(PKV_QP, w1)
                     PKV_R0(PKV_QO, w2)
                 : PKV_S_INOUT(x)
                 : PKV_S_IN, [w0] "v"(r[0]), [w1] "v"(r[1]), [w2] "v"(r[2]));
    roles_turn1(x);
}

// Three rounds whose next K + W words are the partner's ka, own kb, partner's kc: the rounds
// right after a phase barrier, which leave the phase's new words time to arrive from LDS.
__device__ __forceinline__ void pair_r3_pp(uint32_t x[4], uint32_t& q, const PairLane& pl, uint32_t ka, uint32_t kb,
                                          uint32_t kc) {
    uint32_t t0, t1, t2;
    asm volatile(PKV_ALIGN PKV_R0(PKV_QP, w0) PKV_R1(PKV_QO, w1) PKV_R2(PKV_QP, w2)
                 : PKV_S_INOUT(x)
                 : PKV_S_IN, [w0] "v"(ka), [w1] "v"(kb), [w2] "v"(kc));
    roles_turn3(x);
}

// 13 rounds t0 - 1 .. t0 + 11 of a phase whose own words are w (t = t0 + odd + 2j, j = 0..7).
__device__ __forceinline__ void pair_r13_phase(uint32_t x[4], uint32_t& q, const PairLane& pl, const uint32_t w[8]) {
    uint32_t t0, t1, t2;
    asm volatile(PKV_ALIGN PKV_PH4(w0, w1) PKV_PH4(w2, w3) PKV_PH4(w4, w5) PKV_R0(PKV_QO, w6)
                 : PKV_S_INOUT(x)
                 : PKV_S_IN, [w0] "v"(w[0]), [w1] "v"(w[1]), [w2] "v"(w[2]), [w3] "v"(w[3]), [w4] "v"(w[4]),
                   [w5] "v"(w[5]), [w6] "v"(w[6]));
    roles_turn1(x);
}

// Rounds 47..63 of compression 1; the last one forms compression 2's first Q from k2w0 (its
// K_0 + W_0 + h0 on the e lane).
__device__ __forceinline__ void pair_r17_last(uint32_t x[4], uint32_t& q, const PairLane& pl, const uint32_t w[8],
                                             uint32_t k2w0) {
    uint32_t t0, t1, t2;
    asm volatile(PKV_ALIGN PKV_PH4(w0, w1) PKV_PH4(w2, w3) PKV_PH4(w4, w5) PKV_PH4(w6, w7) PKV_R0(PKV_QO, w8)
                 : PKV_S_INOUT(x)
                 : PKV_S_IN, [w0] "v"(w[0]), [w1] "v"(w[1]), [w2] "v"(w[2]), [w3] "v"(w[3]), [w4] "v"(w[4]),
                   [w5] "v"(w[5]), [w6] "v"(w[6]), [w7] "v"(w[7]), [w8] "v"(k2w0));
    roles_turn1(x);
}

// Compression 2 from the chaining value h (read only): 64 rounds whose own K + W words are k
// (t = odd + 2j, j = 0..31), the first four rounds writing fresh registers.
#define PKV_C2_4(KA, KB, KC) PKV_R0(PKV_QP, KA) PKV_R1(PKV_QO, KB) PKV_R2(PKV_QP, KB) PKV_R3(PKV_QO, KC)
__device__ __forceinline__ void pair_c2(uint32_t x[4], uint32_t& q, const PairLane& pl, const uint32_t h[4],
                                       const uint32_t k[32]) {
    uint32_t t0, t1, t2;
    asm volatile(PKV_ALIGN PKV_F0(PKV_QP, k0) PKV_F1(PKV_QO, k1) PKV_F2(PKV_QP, k1) PKV_F3(PKV_QO, k2)
                     PKV_C2_4(k2, k3, k4) PKV_C2_4(k4, k5, k6) PKV_C2_4(k6, k7, k8) PKV_C2_4(k8, k9, k10)
                     PKV_C2_4(k10, k11, k12) PKV_C2_4(k12, k13, k14) PKV_C2_4(k14, k15, k16)
                     PKV_C2_4(k16, k17, k18) PKV_C2_4(k18, k19, k20) PKV_C2_4(k20, k21, k22)
                     PKV_C2_4(k22, k23, k24) PKV_C2_4(k24, k25, k26) PKV_C2_4(k26, k27, k28)
                     PKV_C2_4(k28, k29, k30) PKV_R0(PKV_QP, k30) PKV_R1(PKV_QO, k31) PKV_R2(PKV_QP, k31)
                     PKV_R3(PKV_QN, k31)
                 : PKV_S_FRESH(x)
                 : PKV_S_IN, [i0] "v"(h[0]), [i1] "v"(h[1]), [i2] "v"(h[2]), [i3] "v"(h[3]), [k0] "v"(k[0]),
                   [k1] "v"(k[1]), [k2] "v"(k[2]), [k3] "v"(k[3]), [k4] "v"(k[4]), [k5] "v"(k[5]), [k6] "v"(k[6]),
                   [k7] "v"(k[7]), [k8] "v"(k[8]), [k9] "v"(k[9]), [k10] "v"(k[10]), [k11] "v"(k[11]),
                   [k12] "v"(k[12]), [k13] "v"(k[13]), [k14] "v"(k[14]), [k15] "v"(k[15]), [k16] "v"(k[16]),
                   [k17] "v"(k[17]), [k18] "v"(k[18]), [k19] "v"(k[19]), [k20] "v"(k[20]), [k21] "v"(k[21]),
                   [k22] "v"(k[22]), [k23] "v"(k[23]), [k24] "v"(k[24]), [k25] "v"(k[25]), [k26] "v"(k[26]),
                   [k27] "v"(k[27]), [k28] "v"(k[28]), [k29] "v"(k[29]), [k30] "v"(k[30]), [k31] "v"(k[31]));
}
#undef PKV_C2_4
#undef PKV_S_FRESH
#undef PKV_S_INOUT
#undef PKV_S_IN
#undef PKV_ALIGN
#undef PKV_PH4
#undef PKV_F3
#undef PKV_F2
#undef PKV_F1
#undef PKV_F0
#undef PKV_R3
#undef PKV_R2
#undef PKV_R1
#undef PKV_R0
#undef PKV_SR
#undef PKV_QN
#undef PKV_QP
#undef PKV_QO
#undef PKV_S_HEAD

// Bitwise select m ? a : b in one instruction (v_bfi_b32), with the lane's parity mask m as an
// ordinary register: no condition register to rebuild around each use.
__device__ __forceinline__ uint32_t bsel(uint32_t m, uint32_t a, uint32_t b) {
    uint32_t r;
    asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(m), "v"(a), "v"(b));
    return r;
}

// What a lane of a pair needs for its parity of a message schedule: its parity mask and
// k[j] = K_{2j + odd} for j = 0..31, held in registers for the whole kernel.
struct PairK {
    uint32_t m;
    uint32_t k[32];
};

__device__ __forceinline__ PairK make_pair_k(bool odd) {
    PairK pk;
    pk.m = odd ? ~0u : 0u;
#pragma unroll
    for (int j = 0; j < 32; ++j) pk.k[j] = odd ? kRoundK[2 * j + 1] : kRoundK[2 * j];
    return pk;
}

// One step of a message schedule split over a lane pair: the e lane computes W_{2j}, the a lane
// W_{2j+1}.  v[k] is the lane's own word k+1 steps back.  The e lane needs its partner's
// W_{2j-7} and W_{2j-15}, the a lane its partner's W_{2j-6} and W_{2j-14}; each lane sends
// sigma0 of the older one plus the newer one (z), and adds what its partner sent.  Returns the
// new word and sets wk = word + k.  One asm block of 14 eight-byte instructions, aligned to 8
// bytes (see the rounds above); the partner's z is read by DPP four instructions after it is
// written, so no wait state is needed.
__device__ __forceinline__ uint32_t pair_schedule_step(uint32_t v[8], uint32_t m, uint32_t k, uint32_t& wk) {
    uint32_t w, t0, t1, t2, z;
    asm volatile(".p2align 3\n"
                 "v_bfi_b32 %[t0], %[m], %[v7], %[v6]\n"                  // sigma0 operand
                 "v_alignbit_b32 %[t1], %[t0], %[t0], 7\n"
                 "v_alignbit_b32 %[t2], %[t0], %[t0], 18\n"
                 "v_lshrrev_b32_e64 %[t0], 3, %[t0]\n"
                 "v_bitop3_b32 %[z], %[t1], %[t2], %[t0] bitop3:0x96\n"
                 "v_bfi_b32 %[t0], %[m], %[v3], %[v2]\n"
                 "v_add_u32_e64 %[z], %[z], %[t0]\n"                      // what the partner needs
                 "v_alignbit_b32 %[t1], %[v0], %[v0], 17\n"
                 "v_alignbit_b32 %[t2], %[v0], %[v0], 19\n"
                 "v_lshrrev_b32_e64 %[t0], 10, %[v0]\n"
                 "v_bitop3_b32 %[t1], %[t1], %[t2], %[t0] bitop3:0x96\n"  // sigma1(own word 2 back)
                 "v_add_u32_dpp %[t2], %[z], %[v7] row_ror:8 row_mask:0xf bank_mask:0xf\n"
                 "v_add_u32_e64 %[w], %[t1], %[t2]\n"
                 "v_add_u32_e64 %[wk], %[w], %[k]\n"
                 : [w] "=&v"(w), [wk] "=&v"(wk), [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [z] "=&v"(z)
                 : [m] "v"(m), [v0] "v"(v[0]), [v2] "v"(v[2]), [v3] "v"(v[3]), [v6] "v"(v[6]), [v7] "v"(v[7]),
                   [k] "v"(k));
#pragma unroll
    for (int j = 7; j > 0; --j) v[j] = v[j - 1];
    v[0] = w;
    return w;
}

// Steps j = J0 .. J0+7 of the paired schedule; each lane writes K + W of its word into a column of
// uint4 rows whose first row holds words T0 .. T0+3 (kw1hi: T0 = 16; a token slot: T0 = 0).
template <int J0, int T0 = 16>
__device__ __forceinline__ void pair_schedule8(uint32_t v[8], const PairK& pk, uint32_t* col) {
#pragma unroll
    for (int j = J0; j < J0 + 8; ++j) {
        uint32_t wk;
        pair_schedule_step(v, pk.m, pk.k[j], wk);
        // word t = 2j + odd lives at [(t - T0) / 4][chain].component(t % 4); the lane's column
        // pointer already includes its chain and parity
        col[((2 * j - T0) >> 2) * (kPpChains * 4) + ((2 * j) & 3)] = wk;
    }
}

// The same steps writing K + W in the parity-split layout of PpShared: word t = 2j + odd goes to
// row (t - T0) / 8, component j % 4 of the lane's own parity block (col includes parity and chain).
template <int J0, int T0>
__device__ __forceinline__ void pair_schedule8s(uint32_t v[8], const PairK& pk, uint32_t* col) {
#pragma unroll
    for (int j = J0; j < J0 + 8; ++j) {
        uint32_t wk;
        pair_schedule_step(v, pk.m, pk.k[j], wk);
        col[((2 * j - T0) >> 3) * (kPpChains * 4) + (j & 3)] = wk;
    }
}

// This lane's parity of a key's 16 tokens (out[k] = token 2k + odd), zeros past the chain.
__device__ __forceinline__ void load_tokens_pair(const int32_t* tp, int64_t key, int64_t n, bool odd, uint32_t out[8]) {
    if (key < n) {
        const int32_t* p = tp + key * 16 + (odd ? 1 : 0);
#pragma unroll
        for (int k = 0; k < 8; ++k) out[k] = static_cast<uint32_t>(p[2 * k]);
    } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) out[k] = 0u;
    }
}

// Token-only data of one key (B = 16) by a lane pair: each lane writes its parity of compression
// 1's words 8..15 (and their K + W) and of compression 2's K + W words, computing its parity of
// compression 2's schedule with pair_schedule8.
__device__ __forceinline__ void produce_key_pair(PpShared& sh, uint32_t chain, bool odd, const PairK& pk, int buf,
                                                 const uint32_t tk[8]) {
    const uint32_t o = odd ? 1u : 0u;
    uint32_t* wcol = reinterpret_cast<uint32_t*>(&sh.w1tok[buf][0][chain]) + o;
    uint32_t* kcol = reinterpret_cast<uint32_t*>(&sh.kw1tok[buf][o][chain]);
#pragma unroll
    for (int k = 0; k < 4; ++k) {                      // compression 1, word 8 + 2k + odd = token 2k + odd
        const uint32_t x = bswap(tk[k]);
        const uint32_t kk = pk.k[4 + k];
        wcol[((2 * k) >> 2) * (kPpChains * 4) + ((2 * k) & 3)] = x;
        kcol[k] = x + kk;
    }
    // compression 2: words 0..7 = tokens 8..15, then the padding of a 96-byte message
    uint32_t own[8];
#pragma unroll
    for (int k = 0; k < 4; ++k) own[k] = bswap(tk[4 + k]);
    own[4] = ~pk.m & 0x80000000u;
    own[5] = 0u;
    own[6] = 0u;
    own[7] = pk.m & ((32u + 4u * 16u) * 8u);
    uint32_t* col = reinterpret_cast<uint32_t*>(&sh.kw2[buf][o][0][chain]);
    // word 0 carries h0 as well: the last round of compression 1 forms compression 2's first Q
    // (h of the chaining value + K_0 + W_0) from it
#pragma unroll
    for (int k = 0; k < 8; ++k)
        col[(k >> 2) * (kPpChains * 4) + (k & 3)] = own[k] + pk.k[k] + (k == 0 ? (~pk.m & kInitH[7]) : 0u);
    uint32_t v[8];                                     // own words, newest first
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = own[7 - k];
    pair_schedule8s<8, 0>(v, pk, col);
    pair_schedule8s<16, 0>(v, pk, col);
    pair_schedule8s<24, 0>(v, pk, col);
}

// ---- fused derive and lookup: the helper probes the index while the consumer hashes ------------
// The longest-prefix hit (section 3.4 / 4.1; the hit pkv_lookup_prefix returns) of a chain is
// found by the helper wavefront from the keys the consumer has already produced, so no key makes
// a second trip through HBM and every probe's memory latency hides under the rounds of later keys.
// The two lanes of a chain's pair share the probes: the e lane probes positions 0, 2, 4, .. and
// the a lane positions 1, 3, 5, ..  Once per key period (at the start of the long last phase) a
// lane checks the bucket it loaded one period earlier and then loads the next one: the bucket that
// follows when the checked one is full and neither holds the key nor a never-used slot, else the
// home bucket of its next key.  Two lanes resolve up to two keys per period while the consumer
// produces one, so a chain catches up after probes that continued into a following bucket.  A
// lane stops at its first absent key, and as soon as its partner has found an absent key at a
// smaller position; the hit length is the smaller of the two first absent positions (or the key
// count).  The index is only read, so the caller must not store into it while this runs.
struct PairProbe {
    int64_t next;          // position of the lane's next unresolved key
    int64_t miss;          // position of the lane's first absent key, else the chain's key count
    uint64_t bucket;       // bucket of the probe in flight
    uint64_t visited;      // buckets the probe in flight has checked
    uint4 key;             // key of the probe in flight
    uint4 c[4], p[4];      // its bucket: each slot's {claim word, tag} and {key bytes 8..15, location}
    bool pend;             // a probe is in flight
};

__device__ __forceinline__ void probe_load(const ChainArgs& a, PairProbe& pr) {
    const uint4* q = a.table + pr.bucket * (kBucketWords / 2);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        pr.c[j] = q[2 * j];
        pr.p[j] = q[2 * j + 1];
    }
}

// The first absent position known to the pair (every lane of the wavefront calls this together).
__device__ __forceinline__ int64_t pair_miss(const PairProbe& pr) {
    const uint64_t m = static_cast<uint64_t>(pr.miss);
    const uint64_t other = (static_cast<uint64_t>(lane_swap(static_cast<uint32_t>(m >> 32))) << 32) |
                           lane_swap(static_cast<uint32_t>(m));
    const int64_t o = static_cast<int64_t>(other);
    return o < pr.miss ? o : pr.miss;
}

// One probe point.  Keys 0 .. avail - 1 of the chain exist; `newest` is key period - 1 (the one
// the helper read from LDS this period), every older key is read back from the key array, which
// the consumer wrote at least one workgroup barrier earlier.
__device__ __forceinline__ void probe_point(const ChainArgs& a, PairProbe& pr, int64_t k0, int64_t avail,
                                            int64_t period, uint4 newest) {
    if (pr.pend) {
        const dev::KeyWords kw = dev::key_words(pr.key);
        bool hit = false, empty = false;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            hit |= dev::slot_holds(pr.c[j], pr.p[j], kw);
            empty |= dev::slot_never_used(pr.c[j]);
        }
        ++pr.visited;
        if (hit) {
            pr.next += 2;
            pr.pend = false;
        } else if (empty || pr.visited > a.bucket_mask) {    // a never-used slot, or every bucket checked
            pr.miss = pr.next;
            pr.pend = false;
        } else {
            pr.bucket = (pr.bucket + 1) & a.bucket_mask;
            probe_load(a, pr);
        }
    }
    const int64_t lim = pair_miss(pr);
    if (!pr.pend && pr.next < lim && pr.next < avail) {
        uint4 k = newest;
        if (pr.next != period - 1) k = reinterpret_cast<const uint4*>(a.keys)[k0 + pr.next];
        pr.key = k;
        pr.bucket = dev::home_bucket(pr.key, a.bucket_mask);
        pr.visited = 0;
        probe_load(a, pr);
        pr.pend = true;
    }
}

// P consumer/helper pairs per workgroup (P = 2 puts two consumers on one compute unit, each on its
// own SIMD, when there are enough chains for that); every barrier is workgroup-wide, so all pairs
// run the same number of keys.  FUSED: the helper also finds each chain's hit length (above).
template <int P, bool FUSED>
__global__ __launch_bounds__(kPcThreads * P) void k_derive_b16_pp(ChainArgs a) {
    __shared__ PpShared sh_pairs[P];
    __shared__ int64_t pair_n[2 * P];
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t pair = wave % P;                // consumers are waves 0..P-1, helpers P..2P-1
    PpShared& sh = sh_pairs[pair];
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t c = pair_chain(lane);                   // chain of this lane pair
    const bool odd = pair_is_a(lane);
    const uint32_t base = (blockIdx.x * P + pair) * kPpChains;
    const uint32_t r = base + c;
    int64_t t0 = 0, k0 = 0, n = 0;
    bool valid = r < a.n_req;
    if (valid && !chain_bounds(a, r, t0, k0, n)) valid = false;
    if (!valid) n = 0;
    int64_t nmax = wave_max(n);                 // identical in both wavefronts of a pair
    if (P > 1) {
        if (lane == 0) pair_n[wave] = nmax;
        __syncthreads();
        for (int k = 0; k < 2 * P; ++k) nmax = pair_n[k] > nmax ? pair_n[k] : nmax;
    }
    nmax = uniform64(nmax);
    uint32_t dg[4] = {0u, 0u, 0u, 0u};
    if (valid) load_digest(a, r, dg);

    if (wave < P) {
        // ---------------- consumer: lane pair per chain ----------------
        PairLane pl;
        pl.m = odd ? ~0u : 0u;
        pl.nm = ~pl.m;
        pl.r1 = odd ? 2u : 6u;
        pl.r2 = odd ? 13u : 11u;
        pl.r3 = odd ? 22u : 25u;
        uint32_t iv[4], dgk[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            iv[q] = odd ? kInitH[q] : kInitH[4 + q];
            dgk[q] = dg[q] + kRoundK[4 + q];
        }
        // Q of round 0 of the next key (h0 + K_0 + W_0, e lanes) and K + W of its rounds 1..3
        // (W0..W3 = previous key, held by the a lane and swapped over to the e lane, the only lane
        // whose Q uses them).  The a lanes' Q is zero throughout: every write of Q is masked to the
        // e lanes.
        uint32_t kwp[4], kk[4], key[4] = {0u, 0u, 0u, 0u}, q = odd ? 0u : kRoundK[0] + kInitH[7];
#pragma unroll
        for (int j = 0; j < 4; ++j) kwp[j] = kk[j] = kRoundK[j];
        kk[0] = kRoundK[0] + kInitH[7];
        uint4* const prev_out = &sh.prev[odd ? 1 : 0][c];
        const uint32_t par = odd ? 1u : 0u;
        if (odd) sh.prev[1][c] = make_uint4(0u, 0u, 0u, 0u);
        __syncthreads();                                       // prologue
        for (int64_t i = 0; i < nmax; ++i) {
            const int buf = static_cast<int>(i & 1);
            uint32_t x[4], r1[4], k2[32], wa[8], wb[8], hmid[4];
            if (i > 0) {
                // the previous key, after the barrier that handed it to the helper (its critical
                // path runs from that barrier, this wavefront waits for it at the next one): Q of
                // round 0 and the e lane's K + W of rounds 1..3, and the key into the key array
                swap_q_add3(q, kwp, key, kk);
                if (odd && i - 1 < n)
                    reinterpret_cast<uint4*>(a.keys)[k0 + i - 1] =
                        make_uint4(bswap(key[0]), bswap(key[1]), bswap(key[2]), bswap(key[3]));
            }
            get4(&sh.kw1tok[buf][par][c], r1);
#pragma unroll
            for (int r = 0; r < 8; ++r) get4(&sh.kw2[buf][par][r][c], k2 + 4 * r);
            pair_c1_r0_6(x, q, pl, iv, kwp, dgk);                      // rounds 0..6
            pair_c1_r7_11(x, q, pl, r1);                               // rounds 7..11
            // each phase barrier publishes the helper's next 16 words; the three rounds after it
            // still use the previous words and cover the new ones' LDS latency
            __syncthreads();
            get4(&sh.kw1hi[par][0][c], wa);
            get4(&sh.kw1hi[par][1][c], wa + 4);
            pair_r3_pp(x, q, pl, r1[2], r1[3], r1[3]);                 // rounds 12..14
            pair_r13_phase(x, q, pl, wa);                              // rounds 15..27
            __syncthreads();
            get4(&sh.kw1hi[par][2][c], wb);
            get4(&sh.kw1hi[par][3][c], wb + 4);
            pair_r3_pp(x, q, pl, wa[6], wa[7], wa[7]);                 // rounds 28..30
            pair_r13_phase(x, q, pl, wb);                              // rounds 31..43
            __syncthreads();
            get4(&sh.kw1hi[par][4][c], wa);
            get4(&sh.kw1hi[par][5][c], wa + 4);
            pair_r3_pp(x, q, pl, wb[6], wb[7], wb[7]);                 // rounds 44..46
            pair_r17_last(x, q, pl, wa, k2[0]);                        // rounds 47..63
#pragma unroll
            for (int j = 0; j < 4; ++j) hmid[j] = x[j] + iv[j];
            pair_c2(x, q, pl, hmid, k2);                               // compression 2
#pragma unroll
            for (int j = 0; j < 4; ++j) key[j] = x[j] + hmid[j];   // the key on the a lane
            put4(prev_out, key);
            __syncthreads();                                   // end of key
        }
        if (odd && nmax > 0 && nmax - 1 < n)                   // the last key of a chain of nmax keys
            reinterpret_cast<uint4*>(a.keys)[k0 + nmax - 1] =
                make_uint4(bswap(key[0]), bswap(key[1]), bswap(key[2]), bswap(key[3]));
        __syncthreads();                                       // every key is in the key array
    } else {
        // ---------------- helper: lane pair per chain ----------------
        // The consumer waits at each phase barrier for this wavefront's schedule words, so the
        // helper outranks whatever else shares its SIMD (the index kernels of the previous batch
        // run beside this kernel); it issues little, so the others lose little.
        __builtin_amdgcn_s_setprio(3);
        const int32_t* tp = a.tokens + t0;
        uint32_t dsel[2];
        dsel[0] = odd ? dg[1] : dg[0];     // W4 / W5
        dsel[1] = odd ? dg[3] : dg[2];     // W6 / W7
        uint32_t* kw1hi_col = reinterpret_cast<uint32_t*>(&sh.kw1hi[odd ? 1 : 0][0][c]);
        const PairK pk = make_pair_k(odd);
        uint32_t tk[8], pre[8];
        PairProbe pr;
        if (FUSED) {
            pr.next = odd ? 1 : 0;
            pr.miss = n;
            pr.pend = false;
        }
        load_tokens_pair(tp, 0, n, odd, tk);
        load_tokens_pair(tp, 1, n, odd, pre);
        produce_key_pair(sh, c, odd, pk, 0, tk);
        __syncthreads();                                       // prologue
        for (int64_t i = 0; i < nmax; ++i) {
            const int buf = static_cast<int>(i & 1);
            uint32_t pv[4], tw[8], v[8];
            get4(&sh.prev[1][c], pv);
            get4(&sh.w1tok[buf][0][c], tw);
            get4(&sh.w1tok[buf][1][c], tw + 4);
            // own words, newest first: W14 W12 .. W0 (e lane) or W15 W13 .. W1 (a lane)
#pragma unroll
            for (int k = 0; k < 4; ++k) v[k] = bsel(pk.m, tw[7 - 2 * k], tw[6 - 2 * k]);
            v[4] = dsel[1];
            v[5] = dsel[0];
            v[6] = bsel(pk.m, pv[3], pv[2]);
            v[7] = bsel(pk.m, pv[1], pv[0]);
            pair_schedule8s<8, 16>(v, pk, kw1hi_col);
            __syncthreads();
            pair_schedule8s<16, 16>(v, pk, kw1hi_col);
            __syncthreads();
            pair_schedule8s<24, 16>(v, pk, kw1hi_col);
            __syncthreads();
            if (FUSED) {                                       // keys 0 .. i - 1 exist; pv is key i - 1
                const uint4 newest = make_uint4(bswap(pv[0]), bswap(pv[1]), bswap(pv[2]), bswap(pv[3]));
                probe_point(a, pr, k0, i < n ? i : n, i, newest);
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) tk[q] = pre[q];        // the next key's token-only data
            load_tokens_pair(tp, i + 2, n, odd, pre);
            produce_key_pair(sh, c, odd, pk, buf ^ 1, tk);
            __syncthreads();                                   // end of key
        }
        __syncthreads();                                       // every key is in the key array
        if (FUSED) {
            // every key exists now; finish the probes still open (the exit test is wave-wide, as
            // each probe point exchanges values between the lanes of a pair)
            const uint4 none = make_uint4(0u, 0u, 0u, 0u);
            while (__ballot(pr.pend || pr.next < pair_miss(pr)) != 0) probe_point(a, pr, k0, n, nmax + 1, none);
            const int64_t h = pair_miss(pr);
            if (odd && r < a.n_req) a.hits[r] = static_cast<int32_t>(h);
        }
    }
}

// ---- B = 16m (m >= 2), two wavefronts per 64 chains (used while chains are scarce) -------------
// Same split as for B = 16: the consumer issues only rounds.  Compression 1 of each key (previous
// key | digest | tokens 0..7) runs in four barrier phases while the helper computes its schedule;
// the m token-only compressions that follow (tokens 16c-8 .. 16c+7, the last one padded) are
// produced by the helper two compressions ahead into a ring of three LDS slots, and the consumer
// holds the next compression's 64 K + W words in registers while it runs the current one.
struct PcmShared {
    uint4 kwt[3][16][64];      // K_t + W_t of token-only compressions, three slots
    uint4 w1tok[2][2][64];     // W8..W15 of compression 1 (byte-swapped tokens 0..7), two keys
    uint4 kw1tok[2][2][64];    // K_t + W_t for t = 8..15 of compression 1, two keys
    uint4 kw1hi[12][64];       // K_t + W_t for t = 16..63 of compression 1 (current key)
    uint4 prev[64];            // previous key words (consumer -> helper)
};

// Token words of one production: the 16 (or, for the last compression, 8) words of token
// compression (key, c), and for c == 1 also tokens 0..7 of that key (compression 1's words).
struct Production {
    uint32_t head[8];
    uint32_t w[16];
};

// Where production g sits: key g / m, token compression c = g % m + 1 of that key, ring slot g % 3.
// The loops step it one production at a time (wave-uniform scalars: no division per compression).
struct ProdPos {
    int64_t key;
    uint32_t c;
    uint32_t slot;
};

__device__ __forceinline__ ProdPos prod_pos(int64_t g, uint32_t m) {
    ProdPos p;
    p.key = g / m;
    p.c = static_cast<uint32_t>(g - p.key * m) + 1;
    p.slot = static_cast<uint32_t>(g % 3);
    return p;
}

__device__ __forceinline__ ProdPos prod_next(ProdPos p, uint32_t m) {
    if (p.c == m) {
        p.c = 1;
        ++p.key;
    } else {
        ++p.c;
    }
    p.slot = p.slot == 2 ? 0 : p.slot + 1;
    return p;
}

// Production g (global, g = key * m + (c - 1)) of one lane: compression c (1..m) of `key`.
// Every word is written on every path (zeros past the lane's last key or past the block).
__device__ __forceinline__ void load_production(const int32_t* tp, uint32_t B, uint32_t m, int64_t n,
                                                const ProdPos& at, Production& pr) {
    const int64_t key = at.key;
    const uint32_t c = at.c;
#pragma unroll
    for (int q = 0; q < 8; ++q) pr.head[q] = 0u;
#pragma unroll
    for (int q = 0; q < 16; ++q) pr.w[q] = 0u;
    if (key < n) {
        const int32_t* k = tp + key * static_cast<int64_t>(B);
        if (c == 1) {
#pragma unroll
            for (int q = 0; q < 8; ++q) pr.head[q] = static_cast<uint32_t>(k[q]);
        }
        const int32_t* src = k + 16 * c - 8;
        if (c < m) {
#pragma unroll
            for (int q = 0; q < 16; ++q) pr.w[q] = static_cast<uint32_t>(src[q]);
        } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) pr.w[q] = static_cast<uint32_t>(src[q]);
        }
    }
}

template <typename Shared>
__device__ __forceinline__ void produce_comp(Shared& sh, uint32_t lane, uint32_t m, uint32_t bitlen, const ProdPos& at,
                                             const Production& pr) {
    const int64_t key = at.key;
    const uint32_t c = at.c;
    if (c == 1) {
        const int kb = static_cast<int>(key & 1);
        uint32_t v[8], kv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) { v[q] = bswap(pr.head[q]); kv[q] = v[q] + kRoundK[8 + q]; }
        put4(&sh.w1tok[kb][0][lane], v);
        put4(&sh.w1tok[kb][1][lane], v + 4);
        put4(&sh.kw1tok[kb][0][lane], kv);
        put4(&sh.kw1tok[kb][1][lane], kv + 4);
    }
    uint32_t w[16], kw[16];
    if (c < m) {
#pragma unroll
        for (int q = 0; q < 16; ++q) w[q] = bswap(pr.w[q]);
    } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) w[q] = bswap(pr.w[q]);
        w[8] = 0x80000000u;
#pragma unroll
        for (int q = 9; q < 15; ++q) w[q] = 0u;
        w[15] = bitlen;
    }
    const uint32_t slot = at.slot;
#pragma unroll
    for (int q = 0; q < 16; ++q) kw[q] = w[q] + kRoundK[q];
    lds_put16(&sh.kwt[slot][0], lane, kw);
    schedule16<16>(w, kw);
    lds_put16(&sh.kwt[slot][4], lane, kw);
    schedule16<32>(w, kw);
    lds_put16(&sh.kwt[slot][8], lane, kw);
    schedule16<48>(w, kw);
    lds_put16(&sh.kwt[slot][12], lane, kw);
}

__global__ __launch_bounds__(kPcThreads) void k_derive_m16_pc(ChainArgs a) {
    __shared__ PcmShared sh;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t r = blockIdx.x * 64 + lane;
    const uint32_t B = a.block, m = B / 16;
    const uint32_t bitlen = (32u + 4u * B) * 8u;
    int64_t t0 = 0, k0 = 0, n = 0;
    bool valid = r < a.n_req;
    if (valid && !chain_bounds(a, r, t0, k0, n)) valid = false;
    if (!valid) n = 0;
    const int64_t nmax = wave_max(n);           // identical in both wavefronts
    uint32_t dg[4] = {0u, 0u, 0u, 0u};
    if (valid) load_digest(a, r, dg);
    const int32_t* tp = a.tokens + t0;

    if (wave == 0) {
        // ---------------- consumer ----------------
        uint32_t prev[4] = {0u, 0u, 0u, 0u};
        uint32_t dgk[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) dgk[q] = dg[q] + kRoundK[4 + q];
        put4(&sh.prev[lane], prev);
        __syncthreads();                                       // prologue
        uint32_t slot = 0;                                     // ring slot of the next token compression
        for (int64_t i = 0; i < nmax; ++i) {
            const int kb = static_cast<int>(i & 1);
            uint32_t s[8], h[8], kw[16];
            init_state(s);
#pragma unroll
            for (int q = 0; q < 4; ++q) { kw[q] = prev[q] + kRoundK[q]; kw[4 + q] = dgk[q]; }
            get4(&sh.kw1tok[kb][0][lane], kw + 8);
            get4(&sh.kw1tok[kb][1][lane], kw + 12);
            rounds16(s, kw);                                   // rounds 0..15
            __syncthreads();
            lds_get16(&sh.kw1hi[0], lane, kw);
            rounds16(s, kw);                                   // rounds 16..31
            __syncthreads();
            lds_get16(&sh.kw1hi[4], lane, kw);
            rounds16(s, kw);                                   // rounds 32..47
            __syncthreads();
            lds_get16(&sh.kw1hi[8], lane, kw);
            rounds16(s, kw);                                   // rounds 48..63
#pragma unroll
            for (int q = 0; q < 8; ++q) h[q] = s[q] + kInitH[q];
            __syncthreads();                                   // end of compression 1
            for (uint32_t c = 1; c <= m; ++c) {
                // token compression i * m + c - 1, produced two compressions ago, in ring slot `slot`
                uint32_t kwc[64];
#pragma unroll
                for (int ph = 0; ph < 4; ++ph) lds_get16(&sh.kwt[slot][4 * ph], lane, kwc + 16 * ph);
#pragma unroll
                for (int q = 0; q < 8; ++q) s[q] = h[q];
#pragma unroll
                for (int ph = 0; ph < 4; ++ph) rounds16(s, kwc + 16 * ph);
#pragma unroll
                for (int q = 0; q < 8; ++q) h[q] += s[q];
                if (c == m) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) prev[q] = h[q];
                    if (i < n) store_key(a.keys, k0 + i, prev);
                    put4(&sh.prev[lane], prev);
                }
                __syncthreads();                               // end of token compression c
                slot = slot == 2 ? 0u : slot + 1;
            }
        }
    } else {
        // ---------------- helper ----------------
        Production p0, p1, p2;
        const ProdPos g0 = prod_pos(0, m), g1 = prod_next(g0, m);
        load_production(tp, B, m, n, g0, p0);
        load_production(tp, B, m, n, g1, p1);
        produce_comp(sh, lane, m, bitlen, g0, p0);
        produce_comp(sh, lane, m, bitlen, g1, p1);
        ProdPos make = prod_next(g1, m);                       // production g, made during compression (i, c)
        ProdPos fetch = prod_next(make, m);
        load_production(tp, B, m, n, make, p0);                // p0, p1 = productions g, g + 1
        load_production(tp, B, m, n, fetch, p1);
        fetch = prod_next(fetch, m);                           // production g + 2
        __syncthreads();                                       // prologue
        for (int64_t i = 0; i < nmax; ++i) {
            const int kb = static_cast<int>(i & 1);
            uint32_t w[16], kw[16];
            get4(&sh.prev[lane], w);
#pragma unroll
            for (int q = 0; q < 4; ++q) w[4 + q] = dg[q];
            get4(&sh.w1tok[kb][0][lane], w + 8);
            get4(&sh.w1tok[kb][1][lane], w + 12);
            schedule16<16>(w, kw);
            lds_put16(&sh.kw1hi[0], lane, kw);
            __syncthreads();
            schedule16<32>(w, kw);
            lds_put16(&sh.kw1hi[4], lane, kw);
            __syncthreads();
            schedule16<48>(w, kw);
            lds_put16(&sh.kw1hi[8], lane, kw);
            __syncthreads();
            __syncthreads();                                   // end of compression 1
            for (uint32_t c = 1; c <= m; ++c) {
                p2 = p0;
                p0 = p1;
                load_production(tp, B, m, n, fetch, p1);
                if (make.key < nmax) produce_comp(sh, lane, m, bitlen, make, p2);
                make = prod_next(make, m);
                fetch = prod_next(fetch, m);
                __syncthreads();                               // end of token compression c
            }
        }
    }
}

// ---- B = 16m (m >= 2), each chain on a lane pair (used while chains are very scarce) -----------
// The consumer of k_derive_m16_pc with the lane-pair rounds of k_derive_b16_pp: compression 1 of a
// key runs in four barrier phases while the helper's lane pairs compute its schedule; each of the
// m token-only compressions reads its 64 K + W words from a ring of three LDS slots that the
// helper's lane pairs fill two compressions ahead.
//
// Token words of one production for a lane pair: this lane's parity of the 16 words of token
// compression (key, c) (for the last compression only its 8 token words; the padding is added when
// the words are produced), and for c == 1 its parity of tokens 0..7 (compression 1's words).
// w[k] = word 2k + odd, head[k] = token 2k + odd, not yet byte-swapped; zeros past the chain.
struct PairProduction {
    uint32_t head[4];
    uint32_t w[8];
};

__device__ __forceinline__ void load_production_pair(const int32_t* tp, uint32_t B, uint32_t m, int64_t n,
                                                     const ProdPos& at, bool odd, PairProduction& pr) {
    const int64_t key = at.key;
    const uint32_t c = at.c;
    const uint32_t o = odd ? 1u : 0u;
#pragma unroll
    for (int k = 0; k < 4; ++k) pr.head[k] = 0u;
#pragma unroll
    for (int k = 0; k < 8; ++k) pr.w[k] = 0u;
    if (key < n) {
        const int32_t* kp = tp + key * static_cast<int64_t>(B);
        if (c == 1) {
#pragma unroll
            for (int k = 0; k < 4; ++k) pr.head[k] = static_cast<uint32_t>(kp[2 * k + o]);
        }
        const int32_t* src = kp + 16 * c - 8;
        if (c < m) {
#pragma unroll
            for (int k = 0; k < 8; ++k) pr.w[k] = static_cast<uint32_t>(src[2 * k + o]);
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) pr.w[k] = static_cast<uint32_t>(src[2 * k + o]);
        }
    }
}

// Production g by a lane pair: each lane byte-swaps its parity of the message words, computes its
// parity of the schedule (pair_schedule8) and writes its K + W words into the slot; for c == 1
// also its parity of compression 1's token words.
template <typename Shared>
__device__ __forceinline__ void produce_comp_pair(Shared& sh, uint32_t chain, bool odd, const PairK& pk, uint32_t m,
                                                  uint32_t bitlen, const ProdPos& at, const PairProduction& pr) {
    const int64_t key = at.key;
    const uint32_t c = at.c;
    const uint32_t o = odd ? 1u : 0u;
    if (c == 1) {
        const int kb = static_cast<int>(key & 1);
        uint32_t* wcol = reinterpret_cast<uint32_t*>(&sh.w1tok[kb][0][chain]) + o;
        uint32_t* kcol = reinterpret_cast<uint32_t*>(&sh.kw1tok[kb][0][chain]) + o;
#pragma unroll
        for (int k = 0; k < 4; ++k) {                  // message word 8 + 2k + odd of compression 1
            const uint32_t x = bswap(pr.head[k]);
            const uint32_t kk = pk.k[4 + k];
            wcol[((2 * k) >> 2) * (kPpChains * 4) + ((2 * k) & 3)] = x;
            kcol[((2 * k) >> 2) * (kPpChains * 4) + ((2 * k) & 3)] = x + kk;
        }
    }
    uint32_t own[8];
    if (c < m) {
#pragma unroll
        for (int k = 0; k < 8; ++k) own[k] = bswap(pr.w[k]);
    } else {                                           // words 8..15: 0x80000000, zeros, the bit length
#pragma unroll
        for (int k = 0; k < 4; ++k) own[k] = bswap(pr.w[k]);
        own[4] = ~pk.m & 0x80000000u;
        own[5] = 0u;
        own[6] = 0u;
        own[7] = pk.m & bitlen;
    }
    uint32_t* col = reinterpret_cast<uint32_t*>(&sh.kwt[at.slot][0][chain]) + o;
#pragma unroll
    for (int k = 0; k < 8; ++k) col[((2 * k) >> 2) * (kPpChains * 4) + ((2 * k) & 3)] = own[k] + pk.k[k];
    uint32_t v[8];                                     // own words, newest first
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = own[7 - k];
    pair_schedule8<8, 0>(v, pk, col);
    pair_schedule8<16, 0>(v, pk, col);
    pair_schedule8<24, 0>(v, pk, col);
}

struct PpmShared {
    uint4 kwt[3][16][kPpChains];      // K_t + W_t of token-only compressions, three slots
    uint4 w1tok[2][2][kPpChains];     // W8..W15 of compression 1, two keys
    uint4 kw1tok[2][2][kPpChains];    // K_t + W_t, t = 8..15 of compression 1, two keys
    uint4 kw1hi[12][kPpChains];       // K_t + W_t, t = 16..63 of compression 1 (current key)
    uint4 prev[kPpChains];            // previous key words
};

__global__ __launch_bounds__(kPcThreads) void k_derive_m16_pp(ChainArgs a) {
    __shared__ PpmShared sh;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t c = pair_chain(lane);                   // chain of this lane pair
    const bool odd = pair_is_a(lane);
    const uint32_t r = blockIdx.x * kPpChains + c;
    const uint32_t B = a.block, m = B / 16;
    const uint32_t bitlen = (32u + 4u * B) * 8u;
    int64_t t0 = 0, k0 = 0, n = 0;
    bool valid = r < a.n_req;
    if (valid && !chain_bounds(a, r, t0, k0, n)) valid = false;
    if (!valid) n = 0;
    const int64_t nmax = wave_max(n);           // identical in both wavefronts
    uint32_t dg[4] = {0u, 0u, 0u, 0u};
    if (valid) load_digest(a, r, dg);

    if (wave == 0) {
        // ---------------- consumer: lane pair per chain ----------------
        PairLane pl;
        pl.m = odd ? ~0u : 0u;
        pl.nm = ~pl.m;
        pl.r1 = odd ? 2u : 6u;
        pl.r2 = odd ? 13u : 11u;
        pl.r3 = odd ? 22u : 25u;
        uint32_t iv[4], dgk[4], kwp[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            iv[q] = odd ? kInitH[q] : kInitH[4 + q];
            dgk[q] = dg[q] + kRoundK[4 + q];
            kwp[q] = kRoundK[q];
        }
        if (odd) sh.prev[c] = make_uint4(0u, 0u, 0u, 0u);
        __syncthreads();                                       // prologue
        // K + W of a token compression stream through two 16-word register sets, each block read
        // one block (16 rounds) ahead; the first block of compression g + 1 is read during the last
        // block of compression g (production g + 1 was made during compression g - 1).
        uint32_t kwa[16], kwb[16];
#pragma unroll
        for (int j = 0; j < 4; ++j) get4(&sh.kwt[0][j][c], kwa + 4 * j);
        uint32_t slot = 0;                                     // ring slot of the next token compression
        for (int64_t i = 0; i < nmax; ++i) {
            const int kb = static_cast<int>(i & 1);
            uint32_t x[4], h[4], kw[16], q;
#pragma unroll
            for (int j = 0; j < 4; ++j) { kw[j] = kwp[j]; kw[4 + j] = dgk[j]; }
            get4(&sh.kw1tok[kb][0][c], kw + 8);
            get4(&sh.kw1tok[kb][1][c], kw + 12);
#pragma unroll
            for (int j = 0; j < 4; ++j) x[j] = iv[j];
            q = (x[3] + kw[0]) & pl.nm;
            pair_rounds16_regs(x, q, pl, kw, 0u);               // rounds 0..15
            __syncthreads();
#pragma unroll
            for (int ph = 0; ph < 3; ++ph) {
#pragma unroll
                for (int j = 0; j < 4; ++j) get4(&sh.kw1hi[4 * ph + j][c], kw + 4 * j);
                q = (x[3] + kw[0]) & pl.nm;
                pair_rounds16_regs(x, q, pl, kw, 0u);
                if (ph < 2) __syncthreads();
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) h[j] = x[j] + iv[j];
            __syncthreads();                                   // end of compression 1
            for (uint32_t cc = 1; cc <= m; ++cc) {
                // token compression i * m + cc - 1, produced two compressions ago
                const uint32_t nslot = slot == 2 ? 0u : slot + 1;
#pragma unroll
                for (int j = 0; j < 4; ++j) x[j] = h[j];
                q = (x[3] + kwa[0]) & pl.nm;
#pragma unroll
                for (int j = 0; j < 4; ++j) get4(&sh.kwt[slot][4 + j][c], kwb + 4 * j);
                pair_rounds16_regs(x, q, pl, kwa, kwb[0]);      // rounds 0..15
#pragma unroll
                for (int j = 0; j < 4; ++j) get4(&sh.kwt[slot][8 + j][c], kwa + 4 * j);
                pair_rounds16_regs(x, q, pl, kwb, kwa[0]);      // rounds 16..31
#pragma unroll
                for (int j = 0; j < 4; ++j) get4(&sh.kwt[slot][12 + j][c], kwb + 4 * j);
                pair_rounds16_regs(x, q, pl, kwa, kwb[0]);      // rounds 32..47
#pragma unroll
                for (int j = 0; j < 4; ++j) get4(&sh.kwt[nslot][j][c], kwa + 4 * j);
                pair_rounds16_regs(x, q, pl, kwb, 0u);          // rounds 48..63
#pragma unroll
                for (int j = 0; j < 4; ++j) h[j] += x[j];
                if (cc == m) {                                 // h on the a lane is the key
#pragma unroll
                    for (int j = 0; j < 4; ++j) kwp[j] = lane_swap(h[j]) + kRoundK[j];
                    if (odd) {
                        if (i < n)
                            reinterpret_cast<uint4*>(a.keys)[k0 + i] =
                                make_uint4(bswap(h[0]), bswap(h[1]), bswap(h[2]), bswap(h[3]));
                        put4(&sh.prev[c], h);
                    }
                }
                __syncthreads();                               // end of token compression cc
                slot = nslot;
            }
        }
    } else {
        // ---------------- helper: lane pair per chain ----------------
        const int32_t* tp = a.tokens + t0;
        uint32_t dsel[2];
        dsel[0] = odd ? dg[1] : dg[0];
        dsel[1] = odd ? dg[3] : dg[2];
        uint32_t* kw1hi_col = reinterpret_cast<uint32_t*>(&sh.kw1hi[0][c]) + (odd ? 1 : 0);
        const PairK pk = make_pair_k(odd);
        PairProduction p0, p1, p2;
        const ProdPos g0 = prod_pos(0, m), g1 = prod_next(g0, m);
        load_production_pair(tp, B, m, n, g0, odd, p0);
        load_production_pair(tp, B, m, n, g1, odd, p1);
        produce_comp_pair(sh, c, odd, pk, m, bitlen, g0, p0);
        produce_comp_pair(sh, c, odd, pk, m, bitlen, g1, p1);
        ProdPos make = prod_next(g1, m);                       // production g, made during compression (i, cc)
        ProdPos fetch = prod_next(make, m);
        load_production_pair(tp, B, m, n, make, odd, p0);      // p0, p1 = productions g, g + 1
        load_production_pair(tp, B, m, n, fetch, odd, p1);
        fetch = prod_next(fetch, m);                           // production g + 2
        __syncthreads();                                       // prologue
        for (int64_t i = 0; i < nmax; ++i) {
            const int kb = static_cast<int>(i & 1);
            uint32_t pv[4], tw[8], v[8];
            get4(&sh.prev[c], pv);
            get4(&sh.w1tok[kb][0][c], tw);
            get4(&sh.w1tok[kb][1][c], tw + 4);
#pragma unroll
            for (int k = 0; k < 4; ++k) v[k] = bsel(pk.m, tw[7 - 2 * k], tw[6 - 2 * k]);
            v[4] = dsel[1];
            v[5] = dsel[0];
            v[6] = bsel(pk.m, pv[3], pv[2]);
            v[7] = bsel(pk.m, pv[1], pv[0]);
            pair_schedule8<8>(v, pk, kw1hi_col);
            __syncthreads();
            pair_schedule8<16>(v, pk, kw1hi_col);
            __syncthreads();
            pair_schedule8<24>(v, pk, kw1hi_col);
            __syncthreads();
            __syncthreads();                                   // end of compression 1
            for (uint32_t cc = 1; cc <= m; ++cc) {
                p2 = p0;
                p0 = p1;
                load_production_pair(tp, B, m, n, fetch, odd, p1);
                if (make.key < nmax) produce_comp_pair(sh, c, odd, pk, m, bitlen, make, p2);
                make = prod_next(make, m);
                fetch = prod_next(fetch, m);
                __syncthreads();                               // end of token compression cc
            }
        }
    }
}

// ---- B = 16m, m >= 2: m + 1 compressions per key -------------------------------------------
// Message blocks of one key: block 0 = prev | digest | tokens 0..7; block c (1..m-1) = tokens
// 16c-8 .. 16c+7; block m = tokens 16m-8 .. 16m-1 | padding.  The token words of the next block
// are fetched while the current one is compressed.
__device__ __forceinline__ void load_chunk(const int32_t* tp, uint32_t c, uint32_t m, uint32_t out[16]) {
    if (c == 0) {
#pragma unroll
        for (int q = 0; q < 8; ++q) out[q] = static_cast<uint32_t>(tp[q]);
    } else if (c == m) {
        const int32_t* p = tp + 16 * m - 8;
#pragma unroll
        for (int q = 0; q < 8; ++q) out[q] = static_cast<uint32_t>(p[q]);
    } else {
        const int32_t* p = tp + 16 * c - 8;
#pragma unroll
        for (int q = 0; q < 16; ++q) out[q] = static_cast<uint32_t>(p[q]);
    }
}

__global__ __launch_bounds__(kDeriveThreads) void k_derive_m16(ChainArgs a) {
    const uint32_t r = blockIdx.x * kDeriveThreads + threadIdx.x;
    if (r >= a.n_req) return;
    int64_t t0, k0, n;
    if (!chain_bounds(a, r, t0, k0, n)) return;
    const uint32_t m = a.block / 16;
    const uint32_t bitlen = (32u + 4u * a.block) * 8u;
    uint32_t dg[4], prev[4] = {0u, 0u, 0u, 0u};
    load_digest(a, r, dg);
    const int32_t* base = a.tokens + t0;
    uint32_t nxt[16];
    if (n > 0) load_chunk(base, 0, m, nxt);
    for (int64_t i = 0; i < n; ++i) {
        const int32_t* tp = base + i * a.block;
        uint32_t s[8];
        init_state(s);
        for (uint32_t c = 0; c <= m; ++c) {
            uint32_t cur[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) cur[q] = nxt[q];
            if (c < m) load_chunk(tp, c + 1, m, nxt);
            else if (i + 1 < n) load_chunk(tp + a.block, 0, m, nxt);
            uint32_t w[16];
            if (c == 0) {
#pragma unroll
                for (int q = 0; q < 4; ++q) { w[q] = prev[q]; w[4 + q] = dg[q]; }
#pragma unroll
                for (int q = 0; q < 8; ++q) w[8 + q] = bswap(cur[q]);
            } else if (c == m) {
#pragma unroll
                for (int q = 0; q < 8; ++q) w[q] = bswap(cur[q]);
                w[8] = 0x80000000u;
#pragma unroll
                for (int q = 9; q < 15; ++q) w[q] = 0u;
                w[15] = bitlen;
            } else {
#pragma unroll
                for (int q = 0; q < 16; ++q) w[q] = bswap(cur[q]);
            }
            compress(s, w);
        }
        store_key(a.keys, k0 + i, s);
#pragma unroll
        for (int q = 0; q < 4; ++q) prev[q] = s[q];
    }
}

// ---- any B >= 1: message words selected one by one ------------------------------------------
__global__ __launch_bounds__(kDeriveThreads) void k_derive_any(ChainArgs a) {
    const uint32_t r = blockIdx.x * kDeriveThreads + threadIdx.x;
    if (r >= a.n_req) return;
    int64_t t0, k0, n;
    if (!chain_bounds(a, r, t0, k0, n)) return;
    const uint32_t B = a.block;
    const uint32_t n_blocks = (B + 11u + 15u) / 16u;      // 8 + B message words, 1 pad word, 2 length words
    const uint64_t bitlen = (32ull + 4ull * B) * 8ull;
    uint32_t dg[4], prev[4] = {0u, 0u, 0u, 0u};
    load_digest(a, r, dg);
    for (int64_t i = 0; i < n; ++i) {
        const int32_t* tp = a.tokens + t0 + i * static_cast<int64_t>(B);
        uint32_t s[8];
        init_state(s);
        for (uint32_t c = 0; c < n_blocks; ++c) {
            uint32_t w[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const uint32_t g = 16u * c + q;           // message word index
                const uint32_t ti = g - 8u;               // token index when 8 <= g < 8 + B
                const uint32_t tok = bswap(static_cast<uint32_t>(tp[ti < B ? ti : 0u]));
                uint32_t v = 0u;
                if (g < 4u) v = prev[q & 3];              // only reachable in block 0, q < 4
                else if (g < 8u) v = dg[q & 3];
                else if (ti < B) v = tok;
                else if (g == 8u + B) v = 0x80000000u;
                if (c + 1 == n_blocks) {
                    if (q == 14) v = static_cast<uint32_t>(bitlen >> 32);
                    if (q == 15) v = static_cast<uint32_t>(bitlen);
                }
                w[q] = v;
            }
            compress(s, w);
        }
        store_key(a.keys, k0 + i, s);
#pragma unroll
        for (int q = 0; q < 4; ++q) prev[q] = s[q];
    }
}

// ---- batched descriptor digests: one lane per canonical encoding ----------------------------
// Message word q (big-endian) of a message of L bytes at p with the FIPS 180-4 padding applied
// (bytes past L become 0x80 then zeros), assembled byte by byte: the path for messages that are
// unaligned or empty.
__device__ __forceinline__ uint32_t msg_word_bytes(const uint8_t* p, uint64_t L, uint64_t q) {
    const uint64_t b0 = 4 * q;
    if (b0 >= L) return b0 == L ? 0x80000000u : 0u;
    uint32_t v = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        const uint64_t pos = b0 + b;
        const uint32_t byte = pos < L ? p[pos] : (pos == L ? 0x80u : 0u);
        v = (v << 8) | byte;
    }
    return v;
}


// One message per lane pair, with the derive's paired rounds (the e lane holds e, f, g, h, the a
// lane a, b, c, d).  Both lanes read the block's 16 words; the pair splits the block's schedule
// (even words on the e lane, odd ones on the a lane, pair_schedule_step), and each odd K + W word
// is swapped over to the e lane, which forms Q.  A wavefront holds 32 messages and runs as many
// blocks as its longest message; a pair past its message's last block keeps its state.
//
// The message words come from LDS: the workgroup first copies the byte span of the pool that its
// messages occupy (whole dwords, when it fits the stage) with coalesced loads, so each block costs
// LDS reads instead of a round trip to memory (with one, a block took about 4.5 µs whatever its
// arithmetic).  A word at any byte alignment is two stage dwords and one byte-aligned funnel shift.
// Spans larger than the stage read the pool directly, one block ahead.
constexpr uint32_t kDigestPairs = 32;
constexpr uint32_t kDigestStageWords = 8192;          // 32 KiB

// A message word, big-endian, from its 4 bytes in memory order (le) and the message bytes r it
// holds, clamped to [-1, 4]: 4 keeps it whole, 0..3 keep r bytes and put the 0x80 padding byte
// after them, -1 (past the padding byte) gives 0.
__device__ __forceinline__ uint32_t pad_word(uint32_t le, int32_t r) {
    const uint32_t keep = static_cast<uint32_t>(0xFFFFFFFFull << (8 * (4 - (r > 0 ? r : 0))));
    const uint32_t pad = r >= 0 ? static_cast<uint32_t>(0x80000000ull >> (8 * r)) : 0u;
    return (bswap(le) & keep) | pad;
}

__global__ __launch_bounds__(64) void k_digest_pp(const uint8_t* bytes, uint64_t n_bytes, const int64_t* off,
                                                  const uint32_t* len, uint32_t n, uint8_t* out, int32_t* status) {
    // A batch's digests run beside the previous batch's key derivation and are few wavefronts of
    // serial rounds: without priority, one that shares a SIMD with a round-issuing wavefront only
    // gets the slots that wavefront leaves idle and takes several times as long.
    __builtin_amdgcn_s_setprio(3);
    __shared__ uint32_t stage[kDigestStageWords + 17];   // 17 words of slack: a block's reads are never clamped
    const uint32_t lane = threadIdx.x;
    const uint32_t c = pair_chain(lane);
    const bool odd = pair_is_a(lane);
    const uint32_t i = blockIdx.x * kDigestPairs + c;
    bool valid = i < n;
    int64_t o = 0;
    uint64_t L = 0;
    if (valid) {
        o = off[i];
        L = len[i];
        if (o < 0 || static_cast<uint64_t>(o) > n_bytes || L > n_bytes - static_cast<uint64_t>(o)) {
            dev::report(status, PKV_ELAYOUT);
            valid = false;
        }
    }
    if (!valid) {
        o = 0;
        L = 0;
    }
    const int64_t n_blocks = valid ? static_cast<int64_t>((L + 9 + 63) / 64) : 0;
    const int64_t max_blocks = wave_max(n_blocks);
    const uint64_t bitlen = L * 8;

    // the workgroup's messages as one byte span [lo, hi) of the pool, widened to whole dwords
    const int64_t lo = -wave_max(valid ? -o : -INT64_MAX);
    const int64_t hi = wave_max(valid ? o + static_cast<int64_t>(L) : 0);
    const uintptr_t b0 = reinterpret_cast<uintptr_t>(bytes), pool_end = b0 + n_bytes;
    const uintptr_t s0 = (b0 + static_cast<uintptr_t>(lo)) & ~static_cast<uintptr_t>(3);
    const uint64_t nw = hi > lo ? ((b0 + static_cast<uintptr_t>(hi) + 3) - s0) / 4 : 0;
    const bool staged = nw > 0 && nw <= kDigestStageWords;       // the same on every lane
    if (staged) {
        // Dwords [k_in0, k_in1) lie wholly inside the pool and are copied with unconditional loads,
        // 16 per lane at a time (the index clamped into the range); the span starts at most 3
        // bytes before the pool and ends at most 3 bytes past it, so at most the first and the
        // last dword are assembled from the pool's bytes.
        const uint64_t k_in0 = s0 < b0 ? 1 : 0;
        const uint64_t k_in1 = pool_end >= s0 + 4 ? ((pool_end - s0) / 4 < nw ? (pool_end - s0) / 4 : nw) : 0;
        const uint32_t* s4 = reinterpret_cast<const uint32_t*>(s0);
        if (k_in1 > k_in0) {
            for (uint64_t k0 = k_in0 + lane; k0 < k_in1; k0 += 64 * 16) {
                uint32_t v[16];
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const uint64_t k = k0 + 64 * u;
                    v[u] = s4[k < k_in1 ? k : k_in1 - 1];
                }
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const uint64_t k = k0 + 64 * u;
                    if (k < k_in1) stage[k] = v[u];
                }
            }
        }
        const uint64_t edge = lane == 0 ? 0 : nw - 1;  // lane 0: the first dword, lane 1: the last
        if (lane < 2 && (edge < k_in0 || edge >= k_in1)) {
            const uintptr_t a = s0 + 4 * edge;
            uint32_t v = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (a + j >= b0 && a + j < pool_end) v |= static_cast<uint32_t>(*reinterpret_cast<const uint8_t*>(a + j)) << (8 * j);
            stage[edge] = v;
        }
        // one wavefront: its later LDS reads see these writes
    }
    const uint64_t sb = (b0 + static_cast<uintptr_t>(o)) - s0;    // the message's start in the stage (bytes)
    const uint32_t sh = static_cast<uint32_t>(sb & 3);
    const uint64_t sk = sb >> 2;
    const uint8_t* p = bytes + o;
    const bool fast = L > 0 && (reinterpret_cast<uintptr_t>(p) & 3) == 0 &&
                      static_cast<uint64_t>(o) + ((L + 3) & ~3ull) <= n_bytes;
    const uint32_t* p4 = reinterpret_cast<const uint32_t*>(p);

    // A block's raw words are read one block ahead (into the same registers that the block before
    // has just consumed), then assembled: from the stage, two dwords and a byte-aligned shift per
    // word; from an aligned message, its dwords; otherwise byte by byte.
    const uint64_t flast = fast ? (L - 1) >> 2 : 0;
    PairLane pl;
    pl.m = odd ? ~0u : 0u;
    pl.nm = ~pl.m;
    pl.r1 = odd ? 2u : 6u;
    pl.r2 = odd ? 13u : 11u;
    pl.r3 = odd ? 22u : 25u;
    const PairK pk = make_pair_k(odd);
    uint32_t x[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = odd ? kInitH[q] : kInitH[4 + q];
#define PKV_DIGEST_READ_RAW(BLK)                                                                  \
    do {                                                                                          \
        if (staged) {                                                                             \
            const uint64_t kb64 = sk + 16 * static_cast<uint64_t>(BLK);                           \
            const uint32_t kb = kb64 < kDigestStageWords ? static_cast<uint32_t>(kb64) : kDigestStageWords; \
            _Pragma("unroll") for (int qr = 0; qr < 17; ++qr) raw[qr] = stage[kb + qr];           \
        } else if (fast) {                                                                        \
            _Pragma("unroll") for (int qr = 0; qr < 16; ++qr) {                                   \
                const uint64_t qq = 16 * static_cast<uint64_t>(BLK) + qr;                         \
                raw[qr] = p4[qq < flast ? qq : flast];                                            \
            }                                                                                     \
        }                                                                                         \
    } while (0)
    uint32_t raw[17] = {};
    PKV_DIGEST_READ_RAW(0);
    for (int64_t blk = 0; blk < max_blocks; ++blk) {
        uint32_t w[16], kw[64];
        {
            // message bytes from this block on, clamped: what each word keeps follows from it; a
            // lane past its message (or without one) assembles words that it masks out
            const int64_t rem64 = static_cast<int64_t>(L) - 64 * blk;
            const int32_t rem = static_cast<int32_t>(rem64 < -1 ? -1 : (rem64 > 68 ? 68 : rem64));
            if (staged || fast) {
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const uint32_t le = staged ? __builtin_amdgcn_alignbyte(raw[q + 1], raw[q], sh) : raw[q];
                    const int32_t r = rem - 4 * q;
                    w[q] = pad_word(le, r < -1 ? -1 : (r > 4 ? 4 : r));
                }
            } else {
#pragma unroll
                for (int q = 0; q < 16; ++q) w[q] = msg_word_bytes(p, L, 16 * static_cast<uint64_t>(blk) + q);
            }
            if (blk + 1 == n_blocks) {                 // the last block ends with the bit length
                w[14] = static_cast<uint32_t>(bitlen >> 32);
                w[15] = static_cast<uint32_t>(bitlen);
            }
        }
        if (blk + 1 < max_blocks) PKV_DIGEST_READ_RAW(blk + 1);
#pragma unroll
        for (int t = 0; t < 16; ++t) kw[t] = w[t] + kRoundK[t];
        uint32_t v[8];                                 // own words, newest first (a select per word, not an index)
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = bsel(pk.m, w[15 - 2 * k], w[14 - 2 * k]);
        // the schedule's 16 words for rounds 16 (ph + 1) .. 16 (ph + 1) + 15 are made just before
        // rounds 16 ph .. 16 ph + 15, which need the first of them, so only 32 K + W words are live
        auto schedule16 = [&](int j0) {
#pragma unroll
            for (int j = j0; j < j0 + 8; ++j) {
                uint32_t wk;
                pair_schedule_step(v, pk.m, pk.k[j], wk);
                kw[2 * j] = wk;                        // on the e lane: K + W of round 2j
                kw[2 * j + 1] = lane_swap(wk);         // on the e lane: the a lane's K + W of round 2j + 1
            }
        };
        uint32_t y[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) y[q] = x[q];
        uint32_t q = (y[3] + kw[0]) & pl.nm;
#pragma unroll
        for (int ph = 0; ph < 4; ++ph) {
            if (ph < 3) schedule16(8 + 8 * ph);
            pair_rounds16_regs(y, q, pl, kw + 16 * ph, ph < 3 ? kw[16 * ph + 16] : 0u);
        }
        const bool act = blk < n_blocks;
#pragma unroll
        for (int k = 0; k < 4; ++k) x[k] = act ? x[k] + y[k] : x[k];
    }
    if (valid && odd)                                  // the a lane holds H0..H3
        reinterpret_cast<uint4*>(out)[i] = make_uint4(bswap(x[0]), bswap(x[1]), bswap(x[2]), bswap(x[3]));
}
#undef PKV_DIGEST_READ_RAW

// ---- per-request digests from per-descriptor digests: one lane per request -------------------
__global__ __launch_bounds__(256) void k_expand_digests(const uint4* desc_digests, uint32_t n_desc, const uint32_t* idx,
                                                        uint32_t n_req, uint4* out, int32_t* status) {
    const uint32_t r = blockIdx.x * 256 + threadIdx.x;
    if (r >= n_req) return;
    const uint32_t d = idx[r];
    if (d >= n_desc) {
        dev::report(status, PKV_ELAYOUT);
        out[r] = make_uint4(0u, 0u, 0u, 0u);
        return;
    }
    out[r] = desc_digests[d];
}

// ---- key offsets: floor(len / B) scanned over the requests ------------------------------------
// One workgroup scans a chunk of kScanChunk requests.  A batch of one chunk is done in one launch;
// a larger batch scans every chunk locally (the last entry of each chunk then holds the chunk's
// total), one workgroup turns the chunk ends into global prefix sums, and a last pass adds each
// chunk's offset (the final value at its start) to the rest of the chunk.  The chunk ends double as
// the scratch, so the call needs no memory beyond its output.
constexpr int kScanThreads = 1024;
constexpr int kScanPerThread = 16;
constexpr uint32_t kScanChunk = kScanThreads * kScanPerThread;

// Inclusive scan of per-thread sums across the workgroup: returns this thread's exclusive prefix;
// *total receives the workgroup total.
__device__ __forceinline__ int64_t block_exclusive(int64_t mine, int64_t* wave_sum, int64_t* total) {
    const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int64_t incl = mine;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_up(incl, d, 64);
        if (lane >= static_cast<uint32_t>(d)) incl += y;
    }
    if (lane == 63) wave_sum[wave] = incl;
    __syncthreads();
    int64_t wave_base = 0, t = 0;
    for (uint32_t q = 0; q < kScanThreads / 64; ++q) {
        if (q < wave) wave_base += wave_sum[q];
        t += wave_sum[q];
    }
    *total = t;
    return wave_base + incl - mine;
}

// len / block rounded toward zero, as C's integer division gives it; a power-of-two block (shift >=
// 0 is its log2) takes a shift of the magnitude instead of a 64-bit division.
__device__ __forceinline__ int64_t blocks_of(int64_t len, uint32_t block, int shift) {
    if (shift < 0) return len / block;
    const uint64_t m = len < 0 ? 0ull - static_cast<uint64_t>(len) : static_cast<uint64_t>(len);
    const int64_t q = static_cast<int64_t>(m >> shift);
    return len < 0 ? -q : q;
}

// Chunk blockIdx.x: key_off[r + 1] = sum of floor(len_q / B) over the chunk's requests q <= r.
// The chunk's requests are cut into runs of 64 consecutive ones (lane l takes request l of a run),
// so every load and store of a run is one coalesced 512-byte access; each wavefront scans `runs`
// consecutive runs (as few as cover the chunk, so a small batch spreads over the wavefronts
// instead of queueing on one), chaining their totals, and the wavefronts' totals chain across the
// workgroup.
__global__ __launch_bounds__(kScanThreads) void k_key_offsets(const int64_t* tok_off, uint32_t n_req, uint32_t block,
                                                             int shift, int64_t* key_off) {
    __shared__ int64_t wave_sum[kScanThreads / 64];
    const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (blockIdx.x == 0 && tid == 0) key_off[0] = 0;
    const uint64_t c0 = static_cast<uint64_t>(blockIdx.x) * kScanChunk;
    const uint64_t in_chunk = n_req - c0 < kScanChunk ? n_req - c0 : kScanChunk;
    const uint32_t runs = static_cast<uint32_t>((in_chunk + 64 * (kScanThreads / 64) - 1) / (64 * (kScanThreads / 64)));
    const uint64_t r0 = c0 + static_cast<uint64_t>(wave) * 64 * runs;
    int64_t lo[kScanPerThread], hi[kScanPerThread];
#pragma unroll
    for (int i = 0; i < kScanPerThread; ++i) {            // every boundary the wavefront needs, at once
        const uint64_t r = r0 + 64ull * i + lane;
        const bool in = static_cast<uint32_t>(i) < runs && r < n_req;
        lo[i] = in ? tok_off[r] : 0;
        hi[i] = in ? tok_off[r + 1] : 0;
    }
    int64_t incl[kScanPerThread];
    int64_t run = 0;                                      // the wavefront's total so far
#pragma unroll
    for (int i = 0; i < kScanPerThread; ++i) {
        incl[i] = 0;
        if (static_cast<uint32_t>(i) < runs) {            // uniform across the workgroup
            const uint64_t r = r0 + 64ull * i + lane;
            int64_t x = r < n_req ? blocks_of(hi[i] - lo[i], block, shift) : 0;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int64_t y = __shfl_up(x, d, 64);
                if (lane >= static_cast<uint32_t>(d)) x += y;
            }
            incl[i] = run + x;
            run += __shfl(x, 63, 64);
        }
    }
    if (lane == 0) wave_sum[wave] = run;
    __syncthreads();
    int64_t base = 0;
    for (uint32_t q = 0; q < wave; ++q) base += wave_sum[q];
#pragma unroll
    for (int i = 0; i < kScanPerThread; ++i) {
        const uint64_t r = r0 + 64ull * i + lane;
        if (static_cast<uint32_t>(i) < runs && r < n_req) key_off[r + 1] = base + incl[i];
    }
}

__device__ __forceinline__ uint64_t chunk_end(uint64_t c, uint32_t n_req) {
    const uint64_t e = (c + 1) * kScanChunk;
    return e < n_req ? e : n_req;
}

// One workgroup: the chunk totals at the chunk ends become global prefix sums.
__global__ __launch_bounds__(kScanThreads) void k_key_offsets_carry(uint32_t n_req, int64_t* key_off) {
    __shared__ int64_t wave_sum[kScanThreads / 64];
    __shared__ int64_t carry;
    const uint64_t n_chunks = (static_cast<uint64_t>(n_req) + kScanChunk - 1) / kScanChunk;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (uint64_t t0 = 0; t0 < n_chunks; t0 += kScanThreads) {
        const uint64_t c = t0 + threadIdx.x;
        const int64_t mine = c < n_chunks ? key_off[chunk_end(c, n_req)] : 0;
        int64_t total;
        const int64_t ex = block_exclusive(mine, wave_sum, &total);
        if (c < n_chunks) key_off[chunk_end(c, n_req)] = carry + ex + mine;
        __syncthreads();
        if (threadIdx.x == 0) carry += total;
        __syncthreads();
    }
}

// Chunk blockIdx.x + 1: adds the final value at its start to every entry but its (final) end.
__global__ __launch_bounds__(256) void k_key_offsets_add(uint32_t n_req, int64_t* key_off) {
    const uint64_t c = blockIdx.x + 1ull;
    const uint64_t start = c * kScanChunk, end = chunk_end(c, n_req);
    const int64_t off = key_off[start];
    for (uint64_t i = start + 1 + threadIdx.x; i < end; i += blockDim.x) key_off[i] += off;
}

}  // namespace

// Compute units of the current device, cached per device.  Threads that race on the first call of a
// device all store the same value; the atomics make that well defined.
int compute_units() {
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int cu = cached[dev].load(std::memory_order_relaxed);
    if (cu <= 0) {
        if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cu <= 0) cu = 256;
        cached[dev].store(cu, std::memory_order_relaxed);
    }
    return cu;
}

int launch_derive(const int32_t* tokens, uint64_t n_tokens, const int64_t* tok_off, uint32_t n_req,
                  const uint8_t* digests, uint32_t block, const int64_t* key_off, uint64_t n_keys, uint8_t* keys,
                  int32_t* status, hipStream_t s) {
    if (n_req == 0) return PKV_OK;
    ChainArgs a{tokens, n_tokens, tok_off, n_req, digests, block, key_off, n_keys, keys, status, nullptr, 0, nullptr};
    const dim3 grid((n_req + kDeriveThreads - 1) / kDeriveThreads);
    const unsigned pp_grid = (n_req + kPpChains - 1) / kPpChains;
    const unsigned pp2_grid = (n_req + 2 * kPpChains - 1) / (2 * kPpChains);
    if (block == 16 && pp_grid <= static_cast<unsigned>(compute_units())) {
        hipLaunchKernelGGL((k_derive_b16_pp<1, false>), dim3(pp_grid), dim3(kPcThreads), 0, s, a);
    } else if (block == 16 && pp2_grid <= static_cast<unsigned>(compute_units())) {
        hipLaunchKernelGGL((k_derive_b16_pp<2, false>), dim3(pp2_grid), dim3(2 * kPcThreads), 0, s, a);
    } else if (block == 16) {
        hipLaunchKernelGGL(k_derive_b16, grid, dim3(kDeriveThreads), 0, s, a);
    } else if (block % 16 == 0 && pp_grid <= static_cast<unsigned>(compute_units())) {
        hipLaunchKernelGGL(k_derive_m16_pp, dim3(pp_grid), dim3(kPcThreads), 0, s, a);
    } else if (block % 16 == 0 && grid.x <= static_cast<unsigned>(compute_units())) {
        hipLaunchKernelGGL(k_derive_m16_pc, grid, dim3(kPcThreads), 0, s, a);
    } else if (block % 16 == 0) {
        hipLaunchKernelGGL(k_derive_m16, grid, dim3(kDeriveThreads), 0, s, a);
    } else {
        hipLaunchKernelGGL(k_derive_any, grid, dim3(kDeriveThreads), 0, s, a);
    }
    return check_launch("pkv_derive_keys");
}

// Keys and hit lengths in one kernel where the lane-pair kernel runs the chains (B = 16, at most two
// lane-pair workgroups' chains per compute unit); otherwise the derive and the lookup kernels one
// after the other on the stream.
int launch_derive_lookup(const int32_t* tokens, uint64_t n_tokens, const int64_t* tok_off, uint32_t n_req,
                         const uint8_t* digests, uint32_t block, const int64_t* key_off, uint64_t n_keys,
                         uint8_t* keys, const uint64_t* table, uint64_t capacity, int32_t* hits, int32_t* status,
                         hipStream_t s) {
    if (n_req == 0) return PKV_OK;
    const unsigned pp_grid = (n_req + kPpChains - 1) / kPpChains;
    const unsigned pp2_grid = (n_req + 2 * kPpChains - 1) / (2 * kPpChains);
    const unsigned cus = static_cast<unsigned>(compute_units());
    if (block != 16 || pp2_grid > cus) {
        const int rc = launch_derive(tokens, n_tokens, tok_off, n_req, digests, block, key_off, n_keys, keys, status, s);
        if (rc) return rc;
        return launch_lookup(table, capacity, keys, key_off, n_req, n_keys, hits, nullptr, 0, status, s);
    }
    ChainArgs a{tokens, n_tokens, tok_off, n_req, digests, block, key_off, n_keys, keys, status,
                reinterpret_cast<const uint4*>(table), capacity / kSlotsPerBucket - 1, hits};
    if (pp_grid <= cus)
        hipLaunchKernelGGL((k_derive_b16_pp<1, true>), dim3(pp_grid), dim3(kPcThreads), 0, s, a);
    else
        hipLaunchKernelGGL((k_derive_b16_pp<2, true>), dim3(pp2_grid), dim3(2 * kPcThreads), 0, s, a);
    return check_launch("pkv_derive_lookup");
}

int launch_digest_batch(const uint8_t* bytes, uint64_t n_bytes, const int64_t* off, const uint32_t* len, uint32_t n,
                        uint8_t* out, int32_t* status, hipStream_t s) {
    if (n == 0) return PKV_OK;
    hipLaunchKernelGGL(k_digest_pp, dim3((n + kDigestPairs - 1) / kDigestPairs), dim3(64), 0, s, bytes, n_bytes, off,
                       len, n, out, status);
    return check_launch("pkv_digest_batch");
}

int launch_expand_digests(const uint8_t* desc_digests, uint32_t n_desc, const uint32_t* idx, uint32_t n_req,
                          uint8_t* out, int32_t* status, hipStream_t s) {
    if (n_req == 0) return PKV_OK;
    hipLaunchKernelGGL(k_expand_digests, dim3((n_req + 255) / 256), dim3(256), 0, s,
                       reinterpret_cast<const uint4*>(desc_digests), n_desc, idx, n_req, reinterpret_cast<uint4*>(out),
                       status);
    return check_launch("pkv_expand_digests");
}

int launch_key_offsets(const int64_t* tok_off, uint32_t n_req, uint32_t block, int64_t* key_off, hipStream_t s) {
    const uint64_t n_chunks = (static_cast<uint64_t>(n_req) + kScanChunk - 1) / kScanChunk;
    const int shift = (block & (block - 1)) == 0 ? __builtin_ctz(block) : -1;
    hipLaunchKernelGGL(k_key_offsets, dim3(n_chunks ? static_cast<unsigned>(n_chunks) : 1u), dim3(kScanThreads), 0, s,
                       tok_off, n_req, block, shift, key_off);
    if (n_chunks > 1) {
        hipLaunchKernelGGL(k_key_offsets_carry, dim3(1), dim3(kScanThreads), 0, s, n_req, key_off);
        hipLaunchKernelGGL(k_key_offsets_add, dim3(static_cast<unsigned>(n_chunks - 1)), dim3(256), 0, s, n_req,
                           key_off);
    }
    return check_launch("pkv_key_offsets");
}

}  // namespace pkv
