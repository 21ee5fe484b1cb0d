// hc_device.h -- device-side helpers shared by the gfx950 kernels: the sketch
// hash, cell arithmetic, value types and wave-level utilities.
//
// The sketch format is the one documented in include/hc.h: per batch of c
// parameters (section 3.4) and per hash j < 3 (section 3.1) one 64-bit
// SplitMix64 output gives a row, a rotation and a sign.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hc {

constexpr uint64_t kGolden = 0x9e3779b97f4a7c15ull;   // SplitMix64 increment
constexpr uint64_t kMix1 = 0xbf58476d1ce4e5b9ull;     // SplitMix64 finalizer
constexpr uint64_t kMix2 = 0x94d049bb133111ebull;

// SplitMix64 (Steele, Lea and Flood 2014): output number i of state `seed`.
// The hash helpers are host-callable too: the geometry calls check a blocked
// sketch's seed on the host.
__host__ __device__ __forceinline__ uint64_t splitmix(uint64_t seed, uint64_t i) {
    uint64_t z = seed + (i + 1ull) * kGolden;
    z = (z ^ (z >> 30)) * kMix1;
    z = (z ^ (z >> 27)) * kMix2;
    return z ^ (z >> 31);
}

// Row, rotation and sign of one batch for each of the three hashes.
struct BatchHash {
    uint32_t row[3];
    uint32_t bias[3];
    uint32_t neg;   // bit j set: g_j = -1
};

// floor(a * b / 2^32)
__host__ __device__ __forceinline__ uint32_t mulhi32(uint32_t a, uint32_t b) {
    return (uint32_t)(((uint64_t)a * b) >> 32);
}

// rows: R >= 3 (< 2^32).  cmask = c - 1.
__host__ __device__ __forceinline__ BatchHash batch_hash(uint64_t seed, uint32_t rows,
                                                         uint32_t cmask, uint64_t b) {
    const uint64_t h0 = splitmix(seed, 3ull * b + 0ull);
    const uint64_t h1 = splitmix(seed, 3ull * b + 1ull);
    const uint64_t h2 = splitmix(seed, 3ull * b + 2ull);
    BatchHash h;
    // three distinct rows: scale the low words into [0,R), [0,R-1), [0,R-2)
    // and step later rows over the earlier ones
    uint32_t r0 = mulhi32((uint32_t)h0, rows);
    uint32_t r1 = mulhi32((uint32_t)h1, rows - 1u);
    r1 += (r1 >= r0);
    const uint32_t lo = r0 < r1 ? r0 : r1, hi = r0 < r1 ? r1 : r0;
    uint32_t r2 = mulhi32((uint32_t)h2, rows - 2u);
    r2 += (r2 >= lo);
    r2 += (r2 >= hi);
    h.row[0] = r0;
    h.row[1] = r1;
    h.row[2] = r2;
    h.bias[0] = (uint32_t)(h0 >> 32) & cmask;
    h.bias[1] = (uint32_t)(h1 >> 32) & cmask;
    h.bias[2] = (uint32_t)(h2 >> 32) & cmask;
    h.neg = (uint32_t)(h0 >> 63) | ((uint32_t)(h1 >> 63) << 1) | ((uint32_t)(h2 >> 63) << 2);
    return h;
}

// Counter range of the per-block rotation constants of a blocked sketch: past
// the batch hashes 3b + j (b < 2^32) and the Bloom filter's hashes.
constexpr uint64_t kBlockSaltBase = 1ull << 62;

// P_u(i): a bijection of [0, 2^m), m = 2 log2 c, keyed by u: add s, multiply by
// the odd a1, xor-shift right by h = ceil(m / 2), multiply by the odd a2,
// xor-shift again (each step is invertible modulo 2^m), with a1, a2 and s the
// low, middle and high 20-bit fields of u.
__host__ __device__ __forceinline__ uint32_t block_offsets(uint64_t u, uint32_t i, uint32_t log2c) {
    const uint32_t m = 2u * log2c;
    const uint32_t mask = (1u << m) - 1u;  // m <= 20
    const uint32_t h = (m + 1u) >> 1;
    const uint32_t a1 = ((uint32_t)u & 0xfffffu) | 1u;
    const uint32_t a2 = ((uint32_t)(u >> 20) & 0xfffffu) | 1u;
    const uint32_t s = (uint32_t)(u >> 40) & 0xfffffu;
    uint32_t x = (i + s) & mask;
    x = (x * a1) & mask;
    x ^= x >> h;
    x = (x * a2) & mask;
    x ^= x >> h;
    return x;
}

// Hash of batch b in a blocked sketch, in block-local rows: batch b is number
// i = b mod block of parameter block q = b / block, whose brows rows it draws
// its three distinct rows from (as batch_hash), taken in ascending order.  Its
// first rotation is h_0's; the other two are offset from it by the two base-c
// digits of pi = P_q(i), P_q a bijection of [0, c^2) keyed by the block's
// constant u_q = SplitMix64 output 2^62 + q (block_offsets).  For c >= 32 a
// block's batches (at most 1024 <= c^2) get distinct offset pairs, so no two
// batches of one block can sit on the same three rows with the same relative
// rotations, which would pair every two of their corresponding elements on the
// same three cells (a stopping set that no sketch size peels; with few rows
// per block independent rotations make that likely).  P_q mixes (it is not
// affine in i) so that the offsets carry no arithmetic structure, which would
// itself create small stopping sets.
__host__ __device__ __forceinline__ BatchHash blocked_local_hash(uint64_t seed, uint32_t brows,
                                                                 uint32_t cmask, uint32_t log2c,
                                                                 uint64_t b, uint32_t block) {
    BatchHash h = batch_hash(seed, brows, cmask, b);
    const uint32_t r0 = h.row[0], r1 = h.row[1], r2 = h.row[2];
    const uint32_t lo = r0 < r1 ? (r0 < r2 ? r0 : r2) : (r1 < r2 ? r1 : r2);
    const uint32_t hi = r0 > r1 ? (r0 > r2 ? r0 : r2) : (r1 > r2 ? r1 : r2);
    h.row[0] = lo;
    h.row[1] = r0 + r1 + r2 - lo - hi;
    h.row[2] = hi;
    const uint64_t q = b / block;
    const uint32_t i = (uint32_t)(b - q * block);
    const uint32_t pi = block_offsets(splitmix(seed, kBlockSaltBase + q), i, log2c);
    h.bias[1] = (h.bias[0] + (pi & cmask)) & cmask;
    h.bias[2] = (h.bias[0] + (pi >> log2c)) & cmask;
    return h;
}

// Hash of batch b with global rows: the global sketch's (block == 0), or a
// blocked sketch's local hash offset to the rows of block b / block.
__host__ __device__ __forceinline__ BatchHash batch_hash_blocked(uint64_t seed, uint32_t brows,
                                                                 uint32_t cmask, uint32_t log2c,
                                                                 uint64_t b, uint32_t block) {
    if (block == 0) return batch_hash(seed, brows, cmask, b);
    BatchHash h = blocked_local_hash(seed, brows, cmask, log2c, b, block);
    const uint32_t base = (uint32_t)(b / block) * brows;
    h.row[0] += base;
    h.row[1] += base;
    h.row[2] += base;
    return h;
}

// ---- Bloom-filter index (section 3.3), batched like the sketch (3.4) --------

// Hash i < k of batch b is SplitMix64 output number 3 * 2^32 + k * b + i (a
// counter range the sketch's outputs 3b + j never reach): row
// mulhi32(lo32(u), brows) of the filter's brows rows of c bits, rotation
// (u >> 32) mod c.
constexpr uint64_t kBloomBase = 3ull << 32;

struct BloomHash {
    uint32_t row;
    uint32_t bias;
};

__host__ __device__ __forceinline__ BloomHash bloom_hash(uint64_t seed, uint32_t k,
                                                         uint32_t brows, uint32_t cmask,
                                                         uint64_t b, uint32_t i) {
    const uint64_t u = splitmix(seed, kBloomBase + (uint64_t)k * b + i);
    BloomHash h;
    h.row = mulhi32((uint32_t)u, brows);
    h.bias = (uint32_t)(u >> 32) & cmask;
    return h;
}

// Sets the k filter bits of parameter p: bit row * c + ((t + bias) mod c).
__device__ __forceinline__ void bloom_insert_param(uint32_t* f, uint64_t p, uint64_t seed,
                                                   uint32_t k, uint32_t brows, uint32_t c,
                                                   uint32_t cmask, uint32_t log2c) {
    const uint64_t b = p >> log2c;
    const uint32_t t = (uint32_t)p & cmask;
    for (uint32_t i = 0; i < k; i++) {
        const BloomHash h = bloom_hash(seed, k, brows, cmask, b, i);
        const uint32_t bit = h.row * c + ((t + h.bias) & cmask);
        atomicOr(f + (bit >> 5), 1u << (bit & 31u));
    }
}

// Inserts the nonzeros of one 32-bit mask word (parameters p0 .. p0 + 31, p0 a
// multiple of 32).  For c >= 32 the word lies in one batch and, per hash, its
// bits land rotated in one filter row: at most two filter words receive it, so
// it takes at most 2k atomic ORs whatever its popcount.
__device__ __forceinline__ void bloom_insert_word(uint32_t* f, uint32_t word, uint64_t p0,
                                                  uint64_t seed, uint32_t k, uint32_t brows,
                                                  uint32_t c, uint32_t cmask, uint32_t log2c) {
    if (c >= 32) {
        const uint64_t b = p0 >> log2c;
        const uint32_t cw = c >> 5, ow = ((uint32_t)p0 & cmask) >> 5;
        for (uint32_t i = 0; i < k; i++) {
            const BloomHash h = bloom_hash(seed, k, brows, cmask, b, i);
            const uint32_t q = h.bias >> 5, r = h.bias & 31u;
            uint32_t* rp = f + (uint64_t)h.row * cw;
            const uint32_t w0 = (ow + q) & (cw - 1u);
            const uint32_t lo = word << r;
            if (lo != 0u) atomicOr(rp + w0, lo);
            if (r != 0u) {
                const uint32_t hi = word >> (32u - r);
                if (hi != 0u) atomicOr(rp + ((w0 + 1u) & (cw - 1u)), hi);
            }
        }
    } else {
        while (word != 0u) {
            const uint32_t sbit = (uint32_t)__builtin_ctz(word);
            word &= word - 1u;
            bloom_insert_param(f, p0 + sbit, seed, k, brows, c, cmask, log2c);
        }
    }
}

// Cell of column t under hash j.  c = cmask + 1 is a power of two.
__device__ __forceinline__ uint32_t cell_of(const BatchHash& h, int j, uint32_t t, uint32_t c,
                                            uint32_t cmask) {
    return h.row[j] * c + ((t + h.bias[j]) & cmask);
}

// ---- value types: int32 sums wrap (computed on uint32), fp32 plain ----------

template <typename T> struct Val;

template <> struct Val<int32_t> {
    __device__ __forceinline__ static int32_t sign(int32_t v, bool neg) {
        return neg ? (int32_t)(0u - (uint32_t)v) : v;
    }
    __device__ __forceinline__ static void atomic_add(int32_t* a, int32_t v) {
        atomicAdd(reinterpret_cast<unsigned int*>(a), (unsigned int)v);
    }
    __device__ __forceinline__ static int32_t add(int32_t a, int32_t b) {
        return (int32_t)((uint32_t)a + (uint32_t)b);
    }
    __device__ __forceinline__ static bool nonzero(int32_t v) { return v != 0; }
};

template <> struct Val<float> {
    __device__ __forceinline__ static float sign(float v, bool neg) { return neg ? -v : v; }
    __device__ __forceinline__ static void atomic_add(float* a, float v) {
        unsafeAtomicAdd(a, v);
    }
    __device__ __forceinline__ static float add(float a, float b) { return a + b; }
    __device__ __forceinline__ static bool nonzero(float v) { return v != 0.0f; }
};

template <> struct Val<double> {
    __device__ __forceinline__ static double sign(double v, bool neg) { return neg ? -v : v; }
    __device__ __forceinline__ static void atomic_add(double* a, double v) {
        unsafeAtomicAdd(a, v);
    }
};

// Decode-side arithmetic type: the fp32 variant peels in fp64, so decoding
// adds no rounding of its own beyond the final conversion of each value.
template <typename T> struct Acc { typedef T type; };
template <> struct Acc<float> { typedef double type; };

template <typename T>
__device__ __forceinline__ T median3(T a, T b, T c) {
    const T lo = a < b ? a : b;
    const T hi = a < b ? b : a;
    return c < lo ? lo : (c > hi ? hi : c);
}

// ---- streaming loads through buffer resources --------------------------------

typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));

// Buffer resource over [base, base + bytes), bytes < 2^31 (word 3 as the
// gfx9 family takes it for untyped loads).  Loads through it take a scalar
// base, a scalar offset and a fixed per-lane offset, so the loop that streams
// a gradient keeps no address arithmetic in the vector registers its loads
// write (which would force a full wait on the memory counter at every
// iteration).  Out-of-range addresses read as 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             0x00020000);
}

// 16 bytes at byte offset voff + soff, nontemporal (read once).
template <typename V>
__device__ __forceinline__ V buffer_load16_nt(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                              uint32_t soff) {
    const v4u32 raw = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 2);
    return __builtin_bit_cast(V, raw);
}

// ---- wave64 utilities --------------------------------------------------------

__device__ __forceinline__ uint32_t lane_id() {
    return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

// Number of set bits of `mask` at lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Workgroup barrier that first waits for all of this wave's LDS operations,
// atomics without a return value included.  hipcc does not always emit that
// wait before s_barrier after such atomics (seen on gfx950: a loop of LDS
// float adds followed directly by the barrier), and another wave could then
// read a cell before an add to it has landed.  s_waitcnt 0xc07f is
// lgkmcnt(0) with the vector-memory and export counters left alone.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __syncthreads();
}

// Exclusive scan over the lanes of a workgroup (every lane calls it; s_tmp
// holds one word per wave); *total gets the sum.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* s_tmp,
                                                         uint32_t* total) {
    const uint32_t lane = lane_id();
    const uint32_t wave = threadIdx.x >> 6;
    const uint32_t nwaves = blockDim.x >> 6;
    uint32_t x = v;
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t y = __shfl_up(x, d);
        if (lane >= (uint32_t)d) x += y;
    }
    if (lane == 63) s_tmp[wave] = x;
    lds_barrier();
    uint32_t off = 0, tot = 0;
    for (uint32_t w = 0; w < nwaves; w++) {
        const uint32_t s = s_tmp[w];
        if (w < wave) off += s;
        tot += s;
    }
    lds_barrier();
    *total = tot;
    return off + x - v;
}

__device__ __forceinline__ uint32_t uniform(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

__device__ __forceinline__ uint64_t uniform64(uint64_t v) {
    const uint32_t lo = uniform((uint32_t)v);
    const uint32_t hi = uniform((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// Bits 0..7 of b moved to bits 0, 4, 8, ..., 28.
__device__ __forceinline__ uint32_t spread4(uint32_t b) {
    b &= 0xffu;
    b = (b | (b << 12)) & 0x000f000fu;
    b = (b | (b << 6)) & 0x03030303u;
    b = (b | (b << 3)) & 0x11111111u;
    return b;
}

}  // namespace hc
