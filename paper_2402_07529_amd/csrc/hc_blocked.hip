// hc_blocked.hip -- the blocked sketch of section 3.2 (the Count Sketch split
// into blocks of a fixed size, so that peeling ends in O(1) rounds), encoded
// and decoded with one workgroup per block and the block's sketch in LDS.
//
// Layout: parameter block q holds batches [q*K, (q+1)*K) (K = block, the last
// block may be shorter) and owns sketch rows [q*R_b, (q+1)*R_b).  Every cell an
// element of block q hashes to lies in those rows, so one workgroup builds and
// peels a block's R_b * c cells without touching any other block.
//
// encode  the workgroup zeroes the block's sketch in LDS, streams the block's
//         gradient once (wave tiles of 1024 parameters, four coalesced 16-byte
//         loads per lane, two blocks per CU), writes
//         each tile's 32 bitmap words with one 128-byte store (at the workloads'
//         block densities a third of the words or more are nonzero, and a
//         zero-fill pass plus nonzero-only stores measured slower), adds every
//         nonzero to its three cells with LDS atomics, and
//         stores the finished block sketch with plain coalesced stores: no
//         global atomics and no pre-zeroing of Y.
// decode  the workgroup loads the block's aggregated sketch into LDS as the
//         residual and builds per-cell counters deg * 2^20 + (sum of the
//         members' batch numbers within the block) from the bitmap.  A cell of
//         degree one therefore names its member: the batch, whose hash table
//         entry for the cell's row gives j and the column.  Synchronous peeling
//         rounds (section 3.2) follow, separated by workgroup barriers: in the
//         first half of a round every pure cell checks whether a pure cell of
//         its member with a smaller j exists (the smallest-j rule of the global
//         decode); in the second half the claiming cells recover x = g_j * Y,
//         subtract g * x and the member from its other two cells, and keep
//         their own value, marked as claimed.  The block's dense output,
//         recovered mask and COO entries are then written by the same
//         workgroup: a recovered element finds its value in its claimed cell,
//         an unrecovered one gets the median estimate from the residual.

#include "../../include/hc.h"
#include "hc_device.h"
#include "hc_internal.h"

namespace hc {

namespace {

constexpr int kEncThreads = 1024;
constexpr int kDecThreads = 1024;
constexpr uint32_t kWaveTile = 1024;          // parameters per wave tile (16 per lane)
constexpr uint32_t kDegShift = 20;
constexpr uint32_t kDegOne = 1u << kDegShift;
constexpr uint32_t kSumMask = kDegOne - 1u;
constexpr uint32_t kClaimed = 0x80000000u;
constexpr uint32_t kScratchWords = 64;
constexpr int kAhead = 8;  // global loads a lane keeps in flight in the decode's streaming loops
// members of 64 words from which lanes walk their own words (measured with
// the table entries read once per word: 128 against 512 took the decode of
// BERT-base from 0.253 to 0.240 ms, LSTM 0.157 to 0.154 and VGG19 0.259 to
// 0.256; BERT-base at 5 % is dense either way)
constexpr uint32_t kDenseGroup = 128;

// Control block of the blocked decode (zeroed before the decode kernel).
struct BCtrl {
    unsigned long long support;
    unsigned long long recovered;
    unsigned int rounds;
    unsigned int done;   // workgroups finished
    unsigned int pad[10];
};
static_assert(sizeof(BCtrl) == 64, "blocked control block layout");

// Hash table entry of (batch, j) within a block: local row * c in bits 0..15,
// rotation in bits 16..25, sign in bit 31.
__device__ __forceinline__ uint32_t tab_pack(const BatchHash& h, int j, uint32_t c) {
    return h.row[j] * c | (h.bias[j] << 16) | (((h.neg >> j) & 1u) << 31);
}
__device__ __forceinline__ uint32_t tab_cell(uint32_t e, uint32_t t, uint32_t cmask) {
    return (e & 0xffffu) + ((t + ((e >> 16) & 0x3ffu)) & cmask);
}
__device__ __forceinline__ bool tab_neg(uint32_t e) { return (e >> 31) != 0u; }

struct BlockRange {
    uint64_t b0;   // first batch
    uint64_t p0;   // first parameter
    uint64_t p1;   // one past the last parameter (<= n)
    uint32_t nb;   // batches in the block
};

__device__ __forceinline__ BlockRange block_range(uint32_t q, uint32_t block, uint32_t log2c,
                                                  uint32_t cmask, uint64_t n) {
    BlockRange r;
    r.b0 = (uint64_t)q * block;
    r.p0 = r.b0 << log2c;
    const uint64_t pend = r.p0 + ((uint64_t)block << log2c);
    r.p1 = pend < n ? pend : n;
    r.nb = (uint32_t)((r.p1 - r.p0 + cmask) >> log2c);
    return r;
}

// Local rows, rotations and signs of the block's batches (rows drawn from the
// block's brows rows, section 3.2 blocking of the section 3.1/3.4 hash).
__device__ __forceinline__ void fill_table(uint32_t* s_tab, const BlockRange& r, uint64_t seed,
                                           uint32_t brows, uint32_t c, uint32_t cmask,
                                           uint32_t log2c, uint32_t block) {
    for (uint32_t i = threadIdx.x; i < r.nb; i += blockDim.x) {
        const BatchHash h = blocked_local_hash(seed, brows, cmask, log2c, r.b0 + i, block);
#pragma unroll
        for (int j = 0; j < 3; j++) s_tab[3 * i + j] = tab_pack(h, j, c);
    }
}

template <typename T> struct LdsAdd;
template <> struct LdsAdd<int32_t> {
    __device__ __forceinline__ static void add(int32_t* a, int32_t v) {
        atomicAdd(reinterpret_cast<unsigned int*>(a), (unsigned int)v);
    }
};
template <> struct LdsAdd<float> {
    __device__ __forceinline__ static void add(float* a, float v) { atomicAdd(a, v); }
};
template <> struct LdsAdd<double> {
    __device__ __forceinline__ static void add(double* a, double v) { atomicAdd(a, v); }
};

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d);
    return v;
}

// Sum over the workgroup (every lane gets it).
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* s_tmp) {
    const uint32_t lane = lane_id(), wave = threadIdx.x >> 6, nwaves = blockDim.x >> 6;
    v = wave_sum_u32(v);
    if (lane == 0) s_tmp[wave] = v;
    lds_barrier();
    uint32_t t = 0;
    for (uint32_t w = 0; w < nwaves; w++) t += s_tmp[w];
    lds_barrier();
    return t;
}

// Position of the r-th (0-based) set bit of w; r < popcount(w).
__device__ __forceinline__ uint32_t select_bit(uint32_t w, uint32_t r) {
    uint32_t pos = 0;
#pragma unroll
    for (uint32_t width = 16; width >= 1; width >>= 1) {
        const uint32_t c = __popc(w & ((1u << width) - 1u));
        if (r >= c) {
            r -= c;
            w >>= width;
            pos += width;
        }
    }
    return pos;
}

__device__ __forceinline__ uint32_t load_bword(const uint32_t* b, uint64_t k, uint64_t words,
                                               uint32_t last_mask) {
    if (k >= words) return 0u;
    const uint32_t w = b[k];
    return k == words - 1 ? (w & last_mask) : w;
}

// The same when ok, else 0, with no branch (words >= 1): the load is issued
// at a clamped index and the word masked after it.  A load under a branch was
// followed, inside the branch, by the masking that used it, so the compiler
// waited for a lane's loads one by one instead of keeping kAhead in flight.
__device__ __forceinline__ uint32_t load_bword_nb(const uint32_t* b, uint64_t k, bool ok,
                                                  uint64_t words, uint32_t last_mask) {
    const bool in = ok && k < words;
    const uint32_t w = b[in ? k : 0];
    const uint32_t mask = in ? (k == words - 1 ? last_mask : 0xffffffffu) : 0u;
    return w & mask;
}

// ---- encode ------------------------------------------------------------------

template <typename T>
struct EncArgs {
    const T* x;
    T* y;
    uint32_t* b;
    uint64_t n, seed;
    uint32_t block, brows, bcells, c, cmask, log2c, y_vec, x_vec;
    uint32_t stage_b;  // the block's bitmap words go through LDS (the kernel's SB)
};

// NT threads per workgroup (one block each), D tiles of the gradient in
// flight per wave (D = 1: load, then encode; D >= 2: a rolling pipeline whose
// loads for tile t + (D - 1) waves are issued before tile t is encoded), WPE
// waves per SIMD (the launch bound: 4 leaves 128 VGPRs, 8 leaves 64).  SB: the
// block's bitmap words are staged in LDS and written after the stream.  As a
// compile-time choice it leaves no global store in the streaming loop, so the
// compiler can count the loads in flight exactly: with SB a runtime flag, the
// prefetching loop waited for the next tile's loads too (vmcnt(0)) before
// encoding the current one.  BERT-base at 5 % went from 0.217 to 0.208 ms per
// encode.
template <typename T, int NT, int D, int WPE, bool SB>
__global__ __launch_bounds__(NT, WPE) void encode_blocked_kernel(EncArgs<T> a) {
    extern __shared__ __align__(16) unsigned char lds_raw[];
    T* s_y = reinterpret_cast<T*>(lds_raw);
    uint32_t* s_tab = reinterpret_cast<uint32_t*>(lds_raw + (size_t)a.bcells * sizeof(T));
    uint32_t* s_bm = s_tab + ((3 * a.block + 3) & ~3u);  // staged bitmap words (16-byte aligned)
    const uint32_t q = blockIdx.x;
    const BlockRange r = block_range(q, a.block, a.log2c, a.cmask, a.n);
    for (uint32_t i = threadIdx.x; i < a.bcells; i += NT) s_y[i] = T(0);
    fill_table(s_tab, r, a.seed, a.brows, a.c, a.cmask, a.log2c, a.block);
    lds_barrier();

    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    const uint32_t ntiles = (uint32_t)((r.p1 - r.p0 + kWaveTile - 1) / kWaveTile);
    constexpr uint32_t kWaves = NT / 64;
    typedef T V4 __attribute__((ext_vector_type(4)));
    const uint32_t nfull = a.x_vec ? (uint32_t)((r.p1 - r.p0) / kWaveTile) : 0u;
    // A tile is read as four 16-byte loads per lane: e[l][k] = parameter
    // tp + 256 l + 4 lane + k.  Tiles wholly inside the block (of a
    // dword-aligned gradient) take 16-byte loads through one buffer resource over the
    // block's full tiles (at most 4 MiB; the tile's offset is scalar, the
    // lane's fixed).  A load past the full tiles lies outside the resource and
    // returns zeros without touching memory, so the pipeline issues its loads
    // unconditionally.  The block's last, partial tile reads element by
    // element, zero past the block's end.
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(a.x + r.p0, nfull * (uint32_t)(kWaveTile * sizeof(T)));
    auto load_full = [&](uint32_t tile, T (&e)[4][4]) {
#pragma unroll
        for (int l = 0; l < 4; l++) {
            const V4 v = buffer_load16_nt<V4>(rs, 16u * lane + 1024u * l, tile * (uint32_t)(kWaveTile * sizeof(T)));
            e[l][0] = v.x;
            e[l][1] = v.y;
            e[l][2] = v.z;
            e[l][3] = v.w;
        }
    };
    auto load_part = [&](uint32_t tile, T (&e)[4][4]) {
        const uint64_t tp = r.p0 + (uint64_t)tile * kWaveTile;
#pragma unroll
        for (int l = 0; l < 4; l++)
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const uint64_t p = tp + 256u * l + 4u * lane + k;
                e[l][k] = p < r.p1 ? a.x[p] : T(0);
            }
    };
    auto encode_tile = [&](uint32_t tile, const T (&e)[4][4]) {
        const uint64_t tp = r.p0 + (uint64_t)tile * kWaveTile;
        // bitmap word w = 8 l + i holds parameters 32 w .. 32 w + 31: lanes
        // 8i .. 8i+7 of load l, parameter 4 lane' + k at bit 4 (lane' - 8 i) + k.
        // Load by load, so that only one load's four ballots are live (all
        // sixteen at once made the one-tile kernel at 64 VGPRs spill).
        uint32_t word = 0;
        const uint32_t sh = 8u * (lane & 7u);
#pragma unroll
        for (int l = 0; l < 4; l++) {
            uint64_t m[4];
#pragma unroll
            for (int k = 0; k < 4; k++) m[k] = __ballot(Val<T>::nonzero(e[l][k]));
            if ((lane >> 3) == (uint32_t)l) {
#pragma unroll
                for (int k = 0; k < 4; k++) word |= spread4((uint32_t)(m[k] >> sh)) << k;
            }
            // sketch: three LDS atomics per nonzero
            if ((m[0] | m[1] | m[2] | m[3]) == 0ull) continue;
            const uint64_t lbase = tp + 256u * l;
            if (a.c >= 256) {
                // a load lies in one batch: its table entries are uniform
                const uint32_t bl = uniform((uint32_t)((lbase >> a.log2c) - r.b0));
                const uint32_t e0 = uniform(s_tab[3 * bl]);
                const uint32_t e1 = uniform(s_tab[3 * bl + 1]);
                const uint32_t e2 = uniform(s_tab[3 * bl + 2]);
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    if (!Val<T>::nonzero(e[l][k])) continue;
                    const uint32_t t = ((uint32_t)lbase + 4u * lane + k) & a.cmask;
                    LdsAdd<T>::add(s_y + tab_cell(e0, t, a.cmask), Val<T>::sign(e[l][k], tab_neg(e0)));
                    LdsAdd<T>::add(s_y + tab_cell(e1, t, a.cmask), Val<T>::sign(e[l][k], tab_neg(e1)));
                    LdsAdd<T>::add(s_y + tab_cell(e2, t, a.cmask), Val<T>::sign(e[l][k], tab_neg(e2)));
                }
            } else {
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    if (!Val<T>::nonzero(e[l][k])) continue;
                    const uint64_t p = lbase + 4u * lane + k;
                    const uint32_t bl = (uint32_t)((p >> a.log2c) - r.b0);
                    const uint32_t t = (uint32_t)p & a.cmask;
#pragma unroll
                    for (int j = 0; j < 3; j++) {
                        const uint32_t ee = s_tab[3 * bl + j];
                        LdsAdd<T>::add(s_y + tab_cell(ee, t, a.cmask), Val<T>::sign(e[l][k], tab_neg(ee)));
                    }
                }
            }
        }
        if (lane < 32 && tp + 32ull * lane < r.p1) {
            if (SB)
                s_bm[((tp - r.p0) >> 5) + lane] = word;
            else
                a.b[(tp >> 5) + lane] = word;
        }
    };
    T e[D][4][4];
    if constexpr (D == 1) {
        for (uint32_t tile = wave; tile < nfull; tile += kWaves) {
            load_full(tile, e[0]);
            encode_tile(tile, e[0]);
        }
    } else {
        // rolling pipeline over D register tiles: the loads of tile
        // t + (D - 1) waves are issued before tile t is encoded, every
        // iteration, so the wait before an encode counts exactly the
        // (D - 1) groups issued after its own
#pragma unroll
        for (int k = 0; k + 1 < D; k++) load_full(wave + (uint32_t)k * kWaves, e[k]);
        uint32_t tile = wave;
        for (;;) {
#pragma unroll
            for (int k = 0; k < D; k++) {
                if (tile >= nfull) goto streamed;
                load_full(tile + (uint32_t)(D - 1) * kWaves, e[(k + D - 1) % D]);
                encode_tile(tile, e[k]);
                tile += kWaves;
            }
        }
    streamed:;
    }
    for (uint32_t tile = nfull + wave; tile < ntiles; tile += kWaves) {
        load_part(tile, e[0]);
        encode_tile(tile, e[0]);
    }
    lds_barrier();

    if (SB) {
        // the block's bitmap in one coalesced pass: a global store inside the
        // streaming loop would sit in the memory counter ahead of the next
        // tile's loads, so every iteration would wait for its acknowledgement
        const uint32_t nw = (uint32_t)((r.p1 - r.p0 + 31) >> 5);
        uint32_t* bb = a.b + (r.p0 >> 5);
        if (((reinterpret_cast<uintptr_t>(bb) & 15u) == 0)) {
            const uint32_t nv = nw / 4;
            for (uint32_t i = threadIdx.x; i < nv; i += NT)
                reinterpret_cast<v4u32*>(bb)[i] = reinterpret_cast<const v4u32*>(s_bm)[i];
            for (uint32_t i = 4 * nv + threadIdx.x; i < nw; i += NT) bb[i] = s_bm[i];
        } else {
            for (uint32_t i = threadIdx.x; i < nw; i += NT) bb[i] = s_bm[i];
        }
    }

    T* yb = a.y + (uint64_t)q * a.bcells;
    if (a.y_vec) {
        typedef T V4 __attribute__((ext_vector_type(4)));
        for (uint32_t i = 4u * threadIdx.x; i < a.bcells; i += 4u * NT) {
            const V4 v = {s_y[i], s_y[i + 1], s_y[i + 2], s_y[i + 3]};
            __builtin_nontemporal_store(v, reinterpret_cast<V4*>(yb + i));
        }
    } else {
        for (uint32_t i = threadIdx.x; i < a.bcells; i += NT) yb[i] = s_y[i];
    }
}

// ---- decode ------------------------------------------------------------------

template <typename T>
struct DecArgs {
    const T* y_agg;
    const uint32_t* b;
    const uint32_t* blk;   // support offsets of bitmap chunks (COO output only)
    T* x_out;
    uint32_t* mask;
    uint32_t* coo_idx;
    T* coo_val;
    uint64_t coo_cap;
    BCtrl* bctrl;
    hc_decode_info* info;
    uint64_t n, words, seed;
    uint32_t block, brows, bcells, c, cmask, log2c, last_mask, x_vec;
    uint32_t claim_words;  // int32: words of per-parameter claim bits in LDS (0: none)
};

__global__ void zero_bctrl_kernel(BCtrl* c) {
    if (threadIdx.x < sizeof(BCtrl) / 4) reinterpret_cast<uint32_t*>(c)[threadIdx.x] = 0u;
}

// The member of a degree-one cell i, whose counter names its batch bl: the
// three table entries are loaded together; j is the hash whose row is the
// cell's row, t the member's column.
struct Member {
    uint32_t e[3];
    uint32_t j, t;
};

__device__ __forceinline__ Member member_of(const uint32_t* s_tab, uint32_t bl, uint32_t i,
                                            uint32_t cmask) {
    Member m;
    m.e[0] = s_tab[3 * bl];
    m.e[1] = s_tab[3 * bl + 1];
    m.e[2] = s_tab[3 * bl + 2];
    const uint32_t rowbase = i & ~cmask;
    m.j = (m.e[0] & 0xffffu) == rowbase ? 0u : ((m.e[1] & 0xffffu) == rowbase ? 1u : 2u);
    const uint32_t ej = m.j == 0 ? m.e[0] : (m.j == 1 ? m.e[1] : m.e[2]);
    m.t = ((i & cmask) - ((ej >> 16) & 0x3ffu)) & cmask;
    return m;
}

// Hands the set bits of the lanes' words (one word per lane) out to the
// lanes in order, 64 at a time: f(s, valid, owner, bit) is called by every
// lane of the wave with s = the rank of its bit among all set bits, owner =
// the lane holding it and bit its position (valid = s < total).  Returns the
// number of set bits.  Consecutive lanes get consecutive bits, so the LDS
// accesses of one call hit nearby columns.
template <typename F>
__device__ __forceinline__ uint32_t for_each_set_bit(uint32_t word, F&& f) {
    // exclusive prefix of the lanes' popcounts (0..32, six bits) from one
    // ballot per bit: no cross-lane data movement through LDS
    const uint32_t lane = lane_id();
    const uint32_t cw = __popc(word);
    uint32_t excl = 0, total = 0;
#pragma unroll
    for (int b = 0; b < 6; b++) {
        const uint64_t m = __ballot((cw >> b) & 1u);
        excl += lanes_below(m) << b;
        total += (uint32_t)__popcll(m) << b;
    }
    for (uint32_t s0 = 0; s0 < total; s0 += 64) {
        const uint32_t s = s0 + lane;
        uint32_t lo = 0;
#pragma unroll
        for (uint32_t step = 32; step >= 1; step >>= 1) {
            const uint32_t cand = lo + step;
            if ((uint32_t)__shfl(excl, (int)cand) <= s) lo = cand;
        }
        const uint32_t wrd = (uint32_t)__shfl(word, (int)lo);
        const uint32_t r = s - (uint32_t)__shfl(excl, (int)lo);
        f(s, s < total, lo, select_bit(wrd, r));
    }
    return total;
}

template <typename T>
__global__ __launch_bounds__(kDecThreads) void decode_blocked_kernel(DecArgs<T> a) {
    typedef typename Acc<T>::type A;
    constexpr uint32_t kWaves = kDecThreads / 64;
    extern __shared__ __align__(16) unsigned char lds_raw[];
    const uint32_t bcells = a.bcells;
    A* s_val = reinterpret_cast<A*>(lds_raw);
    uint32_t* s_cnt = reinterpret_cast<uint32_t*>(lds_raw + (size_t)bcells * sizeof(A));
    uint16_t* s_q = reinterpret_cast<uint16_t*>(s_cnt + bcells);  // frontier queue of cells
    uint32_t* s_tab = reinterpret_cast<uint32_t*>(s_q + ((bcells + 1) & ~1u));
    uint32_t* s_tmp = s_tab + 3 * a.block;  // kScratchWords: reductions, wave totals, flags
    uint32_t* s_any = s_tmp + 48;           // a claim was made, by round (parity, or mod 3)
    uint32_t* s_tail = s_tmp + 51;          // queue length
    uint32_t* s_claim = s_tmp + kScratchWords;  // int32 with claim bits: one per block parameter

    const uint32_t q = blockIdx.x;
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = lane_id();
    const uint32_t wave = threadIdx.x >> 6;
    const uint32_t cmask = a.cmask;
    const BlockRange r = block_range(q, a.block, a.log2c, cmask, a.n);

    // residual sketch and counters; kAhead loads in flight per lane (one
    // workgroup per CU leaves no other wave to hide the latency)
    const T* yb = a.y_agg + (uint64_t)q * bcells;
    for (uint32_t k0 = 0; k0 < bcells; k0 += kAhead * kDecThreads) {
        T v[kAhead];
#pragma unroll
        for (int u = 0; u < kAhead; u++) {
            const uint32_t i = k0 + u * kDecThreads + tid;
            v[u] = i < bcells ? yb[i] : T(0);
        }
#pragma unroll
        for (int u = 0; u < kAhead; u++) {
            const uint32_t i = k0 + u * kDecThreads + tid;
            if (i < bcells) {
                s_val[i] = (A)v[u];
                s_cnt[i] = 0u;
            }
        }
    }
    fill_table(s_tab, r, a.seed, a.brows, a.c, cmask, a.log2c, a.block);
    for (uint32_t i = tid; i < a.claim_words; i += kDecThreads) s_claim[i] = 0u;
    if (tid < 4) s_tmp[48 + tid] = 0u;
    lds_barrier();

    // counters from the bitmap.  Wave w takes a contiguous range of groups of
    // 64 words (the output pass below takes the same range, so the support
    // ranks of its COO entries follow from the waves' totals); each lane adds
    // the members of its own word: lanes hold columns 32 apart, which fall on
    // different LDS banks once rotated.
    const uint64_t w0 = r.p0 >> 5;
    const uint64_t w1 = (r.p1 + 31) >> 5;
    const uint32_t ngroups = (uint32_t)((w1 - w0 + 63) >> 6);
    const uint32_t gpw = (ngroups + kWaves - 1) / kWaves;
    const uint32_t g_lo = wave * gpw < ngroups ? wave * gpw : ngroups;
    const uint32_t g_hi = g_lo + gpw < ngroups ? g_lo + gpw : ngroups;
    uint32_t lane_support = 0;
    for (uint32_t ga = g_lo; ga < g_hi; ga += kAhead) {
        uint32_t wv[kAhead];
#pragma unroll
        for (int u = 0; u < kAhead; u++) {
            const uint64_t wi = w0 + 64ull * (ga + u) + lane;
            wv[u] = load_bword_nb(a.b, wi, ga + u < g_hi && wi < w1, a.words, a.last_mask);
        }
#pragma unroll
        for (int u = 0; u < kAhead; u++) {
            const uint64_t pw = (w0 + 64ull * (ga + u) + lane) * 32ull;
            uint32_t word = wv[u];
            lane_support += __popc(word);
            if (a.c >= 32u) {
                // the word's 32 parameters lie in one batch: its three table
                // entries are read once, not once per member
                if (word == 0u) continue;
                const uint32_t bl = (uint32_t)((pw >> a.log2c) - r.b0);
                const uint32_t e0 = s_tab[3 * bl], e1 = s_tab[3 * bl + 1], e2 = s_tab[3 * bl + 2];
                const uint32_t tb = (uint32_t)pw & cmask;
                while (word) {
                    const uint32_t t = tb + (uint32_t)__builtin_ctz(word);
                    word &= word - 1u;
                    atomicAdd(s_cnt + tab_cell(e0, t, cmask), kDegOne + bl);
                    atomicAdd(s_cnt + tab_cell(e1, t, cmask), kDegOne + bl);
                    atomicAdd(s_cnt + tab_cell(e2, t, cmask), kDegOne + bl);
                }
                continue;
            }
            while (word) {
                const uint32_t bit = __builtin_ctz(word);
                word &= word - 1u;
                const uint64_t p = pw + bit;
                const uint32_t bl = (uint32_t)((p >> a.log2c) - r.b0);
                const uint32_t t = (uint32_t)p & cmask;
#pragma unroll
                for (int j = 0; j < 3; j++)
                    atomicAdd(s_cnt + tab_cell(s_tab[3 * bl + j], t, cmask), kDegOne + bl);
            }
        }
    }
    const uint32_t wave_support = wave_sum_u32(lane_support);
    if (lane == 0) s_tmp[32 + wave] = wave_support;
    lds_barrier();

    // round-0 frontier: every cell of degree one, appended to the queue.  A
    // wave counts the pure cells of its own contiguous range of the block's
    // cells (the counters' loads independent of each other), takes their
    // places with one LDS atomic, then writes them: one queue atomic per wave
    // instead of one per wave and step, each waited for in turn
    {
        const uint32_t cpw = (bcells + kWaves * 64u - 1u) / (kWaves * 64u) * 64u;
        const uint32_t lo = wave * cpw < bcells ? wave * cpw : bcells;
        const uint32_t hi = lo + cpw < bcells ? lo + cpw : bcells;
        uint32_t npure = 0;
        for (uint32_t i0 = lo; i0 < hi; i0 += 64u) {
            const uint32_t i = i0 + lane;
            npure += (uint32_t)__popcll(__ballot(i < hi && (s_cnt[i] >> kDegShift) == 1u));
        }
        uint32_t at = 0;
        if (npure != 0u) {
            if (lane == 0) at = atomicAdd(s_tail, npure);
            at = (uint32_t)__builtin_amdgcn_readfirstlane((int)at);
            for (uint32_t i0 = lo; i0 < hi; i0 += 64u) {
                const uint32_t i = i0 + lane;
                const bool pure = i < hi && (s_cnt[i] >> kDegShift) == 1u;
                const uint64_t m = __ballot(pure);
                if (pure) s_q[at + lanes_below(m)] = (uint16_t)i;
                at += (uint32_t)__popcll(m);
            }
        }
    }
    lds_barrier();

    // synchronous peeling rounds (section 3.2).  The frontier of a round is
    // the queue segment [qs, qe): the cells that became pure in the previous
    // round (every cell enters the queue at most once, when its degree reaches
    // one).  Thread t examines entries qs + t, qs + t + 1024, ...; the first
    // half decides, from a state nobody writes, which pure cells recover their
    // member (the smallest j among the member's pure cells); the second half
    // applies them and appends the cells that became pure.
    uint32_t qs = 0, qe = *s_tail;
    uint32_t rounds = 0, recovered = 0;
    // int32 with claim bits: one barrier per round.  Every pure cell of an
    // element holds its value exactly, so whichever frontier entry of the
    // element sets its claim bit first recovers it; the others stand aside,
    // and the elements recovered in a round are still exactly those with a
    // cell in its frontier.  An entry's cell can only lose its member during
    // the round (when another pure cell of the member wins), so an entry that
    // reads it as pure and then loses the claim is the only race, and it is
    // harmless.  The flag of a round lives in slot round mod 3, cleared one
    // round ahead.
    bool single = false;
    if constexpr (std::is_same<T, int32_t>::value) single = a.claim_words != 0u;
    while (single && qs < qe) {
        if (tid == 0) s_any[(rounds + 1u) % 3u] = 0u;
        bool mine = false;
        // every lane of a wave takes the same number of steps, so the cells
        // that became pure are appended with one queue atomic per wave and
        // step; the cell's value is read beside the claim (only the entry that
        // wins the claim uses it, and no other entry changes that cell this
        // round), and the two counter updates go out together
        for (uint32_t base = qs + wave * 64u; base < qe; base += kDecThreads) {
            const uint32_t idx = base + lane;
            bool act = idx < qe;
            const uint32_t cell = s_q[act ? idx : qs];  // a queued cell either way
            const uint32_t cc = s_cnt[cell];
            act = act && (cc >> kDegShift) == 1u;  // else its member left with another cell
            const uint32_t bl = act ? (cc & kSumMask) : 0u;
            const Member m = member_of(s_tab, bl, cell, cmask);
            const A yv = s_val[cell];
            const uint32_t id = bl * a.c + m.t;  // the member's parameter within the block
            const uint32_t bit = 1u << (id & 31u);
            if (act) act = (atomicOr(s_claim + (id >> 5), bit) & bit) == 0u;
            const uint32_t jo0 = m.j == 0 ? 1u : 0u, jo1 = m.j == 2 ? 1u : 2u;
            const uint32_t e0 = jo0 == 0 ? m.e[0] : m.e[1];
            const uint32_t e1 = jo1 == 1 ? m.e[1] : m.e[2];
            const uint32_t c0 = tab_cell(e0, m.t, cmask), c1 = tab_cell(e1, m.t, cmask);
            uint32_t old0 = 0, old1 = 0;
            if (act) {
                mine = true;
                recovered++;
                const uint32_t ej = m.j == 0 ? m.e[0] : (m.j == 1 ? m.e[1] : m.e[2]);
                const A xv = Val<A>::sign(yv, tab_neg(ej));  // x = g_j * Y
                old0 = atomicSub(s_cnt + c0, kDegOne + bl);
                old1 = atomicSub(s_cnt + c1, kDegOne + bl);
                LdsAdd<A>::add(s_val + c0, Val<A>::sign(xv, !tab_neg(e0)));  // -= g * x
                LdsAdd<A>::add(s_val + c1, Val<A>::sign(xv, !tab_neg(e1)));
                s_cnt[cell] = kClaimed | bl;  // keeps g_j * x in s_val[cell]
            }
            const bool p0 = act && (old0 >> kDegShift) == 2u;
            const bool p1 = act && (old1 >> kDegShift) == 2u;
            const uint64_t b0 = __ballot(p0), b1 = __ballot(p1);
            const uint32_t n0 = (uint32_t)__popcll(b0), n = n0 + (uint32_t)__popcll(b1);
            if (n != 0u) {
                uint32_t at = 0;
                if (lane == 0) at = atomicAdd(s_tail, n);
                at = (uint32_t)__builtin_amdgcn_readfirstlane((int)at);
                if (p0) s_q[at + lanes_below(b0)] = (uint16_t)c0;
                if (p1) s_q[at + n0 + lanes_below(b1)] = (uint16_t)c1;
            }
        }
        if (__ballot(mine) != 0ull && lane == 0) s_any[rounds % 3u] = 1u;
        lds_barrier();
        if (s_any[rounds % 3u] == 0u) break;
        rounds++;
        qs = qe;
        qe = *s_tail;
    }
    while (!single && qs < qe) {
        uint32_t claims = 0;  // bit k: entry qs + tid + 1024 k recovers its member
        for (uint32_t k = 0, idx = qs + tid; idx < qe; k++, idx += kDecThreads) {
            const uint32_t cell = s_q[idx];
            const uint32_t cc = s_cnt[cell];
            if ((cc >> kDegShift) != 1u) continue;
            const Member m = member_of(s_tab, cc & kSumMask, cell, cmask);
            bool first = true;
            if (m.j >= 1) first = (s_cnt[tab_cell(m.e[0], m.t, cmask)] >> kDegShift) != 1u;
            if (m.j == 2 && first) first = (s_cnt[tab_cell(m.e[1], m.t, cmask)] >> kDegShift) != 1u;
            if (first) claims |= 1u << k;
        }
        const bool wave_claims = __ballot(claims != 0u) != 0ull;  // every lane takes part
        if (lane == 0 && wave_claims) s_any[rounds & 1u] = 1u;
        lds_barrier();
        if (s_any[rounds & 1u] == 0u) break;
        if (tid == 0) s_any[(rounds + 1u) & 1u] = 0u;
        rounds++;
        while (claims) {
            const uint32_t k = __builtin_ctz(claims);
            claims &= claims - 1u;
            const uint32_t cell = s_q[qs + tid + kDecThreads * k];
            recovered++;
            const uint32_t bl = s_cnt[cell] & kSumMask;
            const Member m = member_of(s_tab, bl, cell, cmask);
            const uint32_t ej = m.j == 0 ? m.e[0] : (m.j == 1 ? m.e[1] : m.e[2]);
            const A xv = Val<A>::sign(s_val[cell], tab_neg(ej));  // x = g_j * Y
#pragma unroll
            for (uint32_t jj = 0; jj < 3; jj++) {
                if (jj == m.j) continue;
                const uint32_t c2 = tab_cell(m.e[jj], m.t, cmask);
                const uint32_t old = atomicSub(s_cnt + c2, kDegOne + bl);
                if ((old >> kDegShift) == 2u) s_q[atomicAdd(s_tail, 1u)] = (uint16_t)c2;
                LdsAdd<A>::add(s_val + c2, Val<A>::sign(xv, !tab_neg(m.e[jj])));  // -= g * x
            }
            s_cnt[cell] = kClaimed | bl;  // keeps g_j * x in s_val[cell]
        }
        lds_barrier();
        qs = qe;
        qe = *s_tail;
    }
    recovered = block_sum(recovered, s_tmp);

    uint32_t sup_total = 0, wave_rank = 0;
    for (uint32_t w = 0; w < kWaves; w++) {
        const uint32_t s = s_tmp[32 + w];
        if (w < wave) wave_rank += s;
        sup_total += s;
    }

    // outputs, wave w over its range of word groups again (64 words, 2048
    // parameters).  The members of a group are handed out to the lanes in
    // order; each finds its value -- in its claimed cell, or the median
    // estimate from the residual if it was not recovered -- and leaves it in
    // the wave's staging slots (the queue's LDS, free now) at its rank in the
    // group, with its COO entry at its support rank.  The group's dense output
    // is then written as 16-byte vectors, each lane taking 4 parameters and
    // their values from the staging slots by rank.  A group with more members
    // than a wave's slots stores its values directly.
    const bool want_coo = a.coo_idx != nullptr;
    uint64_t rank = 0;
    if (want_coo) {
        const uint64_t chunk = w0 / kChunkWords;
        uint32_t part = 0;
        for (uint64_t w = chunk * kChunkWords + tid; w < w0; w += kDecThreads)
            part += __popc(load_bword(a.b, w, a.words, a.last_mask));
        rank = (uint64_t)a.blk[chunk] + block_sum(part, s_tmp) + wave_rank;
    }
    const uint32_t slots = (((bcells + 1) & ~1u) / 2) / kWaves;  // u32 slots per wave
    T* s_stage = reinterpret_cast<T*>(s_q) + wave * slots;
    typedef T V4 __attribute__((ext_vector_type(4)));
    for (uint32_t ga = g_lo; ga < g_hi; ga += kAhead) {
        uint32_t wv[kAhead];
#pragma unroll
        for (int u = 0; u < kAhead; u++) {
            const uint64_t wi2 = w0 + 64ull * (ga + u) + lane;
            wv[u] = load_bword_nb(a.b, wi2, ga + u < g_hi && wi2 < w1, a.words, a.last_mask);
        }
#pragma unroll
        for (int u = 0; u < kAhead; u++) {
            if (ga + u >= g_hi) break;  // uniform over the wave
            const uint64_t base = w0 + 64ull * (ga + u);
            const uint32_t word = wv[u];
            if (a.mask != nullptr && base + lane < w1) a.mask[base + lane] = word;
            // rank of the first member of each word within the group
            const uint32_t cw = __popc(word);
            uint32_t excl = 0, total = 0;
#pragma unroll
            for (int b = 0; b < 6; b++) {
                const uint64_t mb = __ballot((cw >> b) & 1u);
                excl += lanes_below(mb) << b;
                total += (uint32_t)__popcll(mb) << b;
            }
            // member p (of batch bl, whose table entries are e) takes its
            // value from its claimed cell, or the median estimate
            auto member_e = [&](uint32_t s, bool valid, uint64_t p, uint32_t bl,
                                const uint32_t (&ee)[3]) {
                A val = A(0);
                bool found = true;
                if (valid) {
                    const uint32_t t = (uint32_t)p & cmask;
                    A est[3];
                    found = false;
#pragma unroll
                    for (int j = 0; j < 3; j++) {
                        const uint32_t e = ee[j];
                        const uint32_t cell = tab_cell(e, t, cmask);
                        est[j] = Val<A>::sign(s_val[cell], tab_neg(e));
                        if (s_cnt[cell] == (kClaimed | bl)) {
                            val = est[j];
                            found = true;
                        }
                    }
                    if (!found) val = median3(est[0], est[1], est[2]);
                    const T out = (T)val;
                    if (s < slots) s_stage[s] = out;
                    else if (a.x_out != nullptr) a.x_out[p] = out;
                    if (want_coo) {
                        const uint64_t rr = rank + s;
                        if (rr < a.coo_cap) {
                            a.coo_idx[rr] = (uint32_t)p;
                            a.coo_val[rr] = out;
                        }
                    }
                }
                // members left unrecovered (failed blocks only) leave the mask
                if (a.mask != nullptr && __ballot(!found) != 0ull) {
                    __threadfence_block();  // the plain mask stores above land first
                    if (!found) atomicAnd(a.mask + (p >> 5), ~(1u << (p & 31u)));
                }
            };
            auto member = [&](uint32_t s, bool valid, uint32_t owner, uint32_t bit) {
                const uint64_t p = (base + owner) * 32ull + bit;
                const uint32_t bl = valid ? (uint32_t)((p >> a.log2c) - r.b0) : 0u;
                const uint32_t ee[3] = {s_tab[3 * bl], s_tab[3 * bl + 1], s_tab[3 * bl + 2]};
                member_e(s, valid, p, bl, ee);
            };
            if (total >= kDenseGroup) {
                // a dense group: each lane walks its own word's members (no
                // search across lanes for every member; measured on a 73 %
                // dense BERT-base aggregate).  For c >= 32 the word lies in
                // one batch, whose table entries are read once.
                uint32_t bits = word, rk = 0;
                if (a.c >= 32u) {
                    const uint64_t pw = (base + lane) * 32ull;
                    const uint32_t blw = word != 0u ? (uint32_t)((pw >> a.log2c) - r.b0) : 0u;
                    const uint32_t ew[3] = {s_tab[3 * blw], s_tab[3 * blw + 1], s_tab[3 * blw + 2]};
                    while (bits != 0u) {
                        const uint32_t bit = (uint32_t)__builtin_ctz(bits);
                        bits &= bits - 1u;
                        member_e(excl + rk, true, pw + bit, blw, ew);
                        rk++;
                    }
                }
                while (bits != 0u) {
                    const uint32_t bit = (uint32_t)__builtin_ctz(bits);
                    bits &= bits - 1u;
                    member(excl + rk, true, lane, bit);
                    rk++;
                }
            } else {
                for_each_set_bit(word, member);
            }
            rank += total;
            if (a.x_out != nullptr) {
#pragma unroll
                for (int k = 0; k < 8; k++) {
                    const uint32_t off = 256u * k + 4u * lane;  // parameter offset in the group
                    const uint32_t gw = (uint32_t)__shfl(word, (int)(off >> 5));
                    const uint32_t ge = (uint32_t)__shfl(excl, (int)(off >> 5));
                    const uint64_t pp = base * 32ull + off;
                    if (pp >= r.p1) continue;
                    const uint32_t sh = off & 31u;
                    const uint32_t bits = (gw >> sh) & 0xfu;
                    uint32_t rk = ge + __popc(gw & ((1u << sh) - 1u));  // rank of the first member
                    T v[4];
                    bool stored[4];  // value already stored directly (past the slots)
                    bool any_stored = false;
#pragma unroll
                    for (int kk = 0; kk < 4; kk++) {
                        v[kk] = T(0);
                        stored[kk] = false;
                        if ((bits >> kk) & 1u) {
                            if (rk < slots) v[kk] = s_stage[rk];
                            else stored[kk] = true;
                            rk++;
                        }
                        any_stored |= stored[kk];
                    }
                    if (!any_stored && a.x_vec && pp + 4 <= a.n) {
                        const V4 z = {v[0], v[1], v[2], v[3]};
                        __builtin_nontemporal_store(z, reinterpret_cast<V4*>(a.x_out + pp));
                    } else {
#pragma unroll
                        for (int kk = 0; kk < 4; kk++)
                            if (!stored[kk] && pp + kk < a.n) a.x_out[pp + kk] = v[kk];
                    }
                }
            }
        }
    }

    // block totals; the last workgroup to finish writes the summary.  The
    // totals are atomics and are read back with coherent loads, so the ticket
    // only has to follow them (s_waitcnt 0): an agent-scope fence here wrote
    // back and invalidated the XCD's L2 at the end of every block, with the
    // block's dense output still in it
    if (tid == 0) {
        atomicAdd(&a.bctrl->support, (unsigned long long)sup_total);
        atomicAdd(&a.bctrl->recovered, (unsigned long long)recovered);
        atomicMax(&a.bctrl->rounds, rounds);
        __builtin_amdgcn_s_waitcnt(0);
        const uint32_t ticket = atomicAdd(&a.bctrl->done, 1u);
        if (ticket == gridDim.x - 1) {
            const unsigned long long sup =
                __hip_atomic_load(&a.bctrl->support, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const unsigned long long rec =
                __hip_atomic_load(&a.bctrl->recovered, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const unsigned int rnd =
                __hip_atomic_load(&a.bctrl->rounds, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            a.info->n_support = sup;
            a.info->n_recovered = rec;
            a.info->rounds = rnd;
            a.info->success = rec == sup ? 1u : 0u;
            a.info->status = 0u;
        }
    }
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

template <typename K>
hipError_t allow_lds(K kernel) {
    return allow_dynamic_lds(reinterpret_cast<const void*>(kernel),
                             (int)(kLdsBytes - kLdsReserve));
}

template <typename T>
hipError_t launch_encode_blocked_t(const Geo& g, const void* x, void* y, uint32_t* b,
                                   hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    const bool pf = g.nblocks <= 2u * (uint32_t)di.cus;
    EncArgs<T> a;
    a.x = static_cast<const T*>(x);
    a.y = static_cast<T*>(y);
    a.b = b;
    a.n = g.n;
    a.seed = g.seed;
    a.block = g.block;
    a.brows = g.brows;
    a.bcells = g.brows * g.c;
    a.c = g.c;
    a.cmask = g.cmask;
    a.log2c = g.log2c;
    a.y_vec = (reinterpret_cast<uintptr_t>(y) & 15u) == 0 && (a.bcells & 3u) == 0;
    // the 16-byte buffer loads serve any dword-aligned gradient (every valid
    // one), also off the 16-byte grid: such a view took the element-wise loads
    // before, 105 against 69 us per call on an LSTM-sized block
    a.x_vec = (reinterpret_cast<uintptr_t>(x) & 3u) == 0;
    // stage the bitmap in LDS when two blocks per CU still fit
    const size_t lds = blocked_encode_lds(g);
    const size_t staged = lds + 16 + (size_t)g.block * g.c / 8;
    a.stage_b = staged + kLdsReserve <= kLdsBytes / 2 ? 1u : 0u;
    // the variants as compile-time choices: with the bitmap staged in LDS the
    // streaming loop issues no global stores, so the compiler's load waits
    // count exactly the loads it has in flight
    auto launch = [&](auto kernel, int nt) -> hipError_t {
        hipError_t err = allow_lds(kernel);
        if (err != hipSuccess) return err;
        hipLaunchKernelGGL(kernel, dim3(g.nblocks), dim3(nt), a.stage_b ? staged : lds, s, a);
        return hipGetLastError();
    };
    // Variants measured on MI355X (blocked encode per call; int32 at 1 %):
    // 512 lanes with a two-tile pipeline, two blocks per CU: BERT-base 0.098
    // -> 0.094 ms, VGG19 0.127 -> 0.121 ms, LSTM 0.093 -> 0.088 ms against
    // the best of the 1024-lane ones.  Deeper pipelines (three or four tiles)
    // and 256-lane workgroups were slower.  fp32 (LDS float atomics, whose
    // latency more waves hide better), blocks too large for two per CU, and
    // blocks of few tiles (BERT-base at 5 %: 16 tiles of c = 32 batches, where
    // the block's setup and sketch write-back weigh most and 1024 lanes share
    // them: 0.194 against 0.209 ms) keep 1024 lanes: one tile per wave when
    // there are more than two blocks per CU to run, else a two-tile pipeline.
    const size_t lds_used = a.stage_b ? staged : lds;
    const bool two_per_cu = lds_used + kLdsReserve <= kLdsBytes / 2;
    const uint64_t block_tiles = ((uint64_t)g.block * g.c) / kWaveTile;
#define HC_ENC_SEL(NT, D, WPE)                                                       \
    return a.stage_b ? launch(&encode_blocked_kernel<T, NT, D, WPE, true>, NT)      \
                     : launch(&encode_blocked_kernel<T, NT, D, WPE, false>, NT)
    if (!g.f32 && two_per_cu && block_tiles >= 64) HC_ENC_SEL(512, 2, 4);
    if (pf) HC_ENC_SEL(1024, 2, 4);
    HC_ENC_SEL(1024, 1, 8);
#undef HC_ENC_SEL
}

template <typename T>
hipError_t launch_decode_blocked_t(const Geo& g, const void* y_agg, const uint32_t* b,
                                   const DecodeOut& out, const BlockedLayout& L, void* ws,
                                   hipStream_t s) {
    hipError_t e = allow_lds(&decode_blocked_kernel<T>);
    if (e != hipSuccess) return e;
    char* base = static_cast<char*>(ws);
    BCtrl* bctrl = reinterpret_cast<BCtrl*>(base + L.bctrl);
    uint32_t* blk = reinterpret_cast<uint32_t*>(base + L.blk);
    hipLaunchKernelGGL(zero_bctrl_kernel, dim3(1), dim3(64), 0, s, bctrl);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    DecArgs<T> a;
    a.coo_cap = out.coo_idx != nullptr && out.coo_val != nullptr ? out.coo_cap : 0;
    a.coo_idx = a.coo_cap ? out.coo_idx : nullptr;
    a.coo_val = a.coo_cap ? static_cast<T*>(out.coo_val) : nullptr;
    if (a.coo_idx != nullptr) {
        e = launch_support_offsets(g, b, blk, base + L.ctrl, s);
        if (e != hipSuccess) return e;
    }
    a.y_agg = static_cast<const T*>(y_agg);
    a.b = b;
    a.blk = blk;
    a.x_out = static_cast<T*>(out.x_out);
    a.mask = out.mask;
    a.bctrl = bctrl;
    a.info = static_cast<hc_decode_info*>(out.info);
    a.n = g.n;
    a.words = g.words;
    a.seed = g.seed;
    a.block = g.block;
    a.brows = g.brows;
    a.bcells = g.brows * g.c;
    a.c = g.c;
    a.cmask = g.cmask;
    a.log2c = g.log2c;
    a.last_mask = (g.n & 31u) ? ((1u << (g.n & 31u)) - 1u) : 0xffffffffu;
    a.x_vec = (reinterpret_cast<uintptr_t>(out.x_out) & 15u) == 0;
    // int32: claim bits for the block's parameters when they fit beside the
    // block's sketch (one barrier per peeling round instead of two)
    size_t lds = blocked_decode_lds(g);
    const uint32_t claim_words = (uint32_t)(((size_t)g.block * g.c + 31) / 32);
    a.claim_words = 0;
    if (!g.f32 && lds + (size_t)claim_words * 4 + kLdsReserve <= kLdsBytes) {
        a.claim_words = claim_words;
        lds += (size_t)claim_words * 4;
    }
    hipLaunchKernelGGL(decode_blocked_kernel<T>, dim3(g.nblocks), dim3(kDecThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace

size_t blocked_encode_lds(const Geo& g) {
    return (size_t)g.brows * g.c * 4 + (size_t)g.block * 12;
}

size_t blocked_decode_lds(const Geo& g) {
    const size_t vsz = g.f32 ? 8 : 4;  // residual: int32, or fp64 for fp32 gradients
    const size_t cells = (size_t)g.brows * g.c;
    // residual + counters + frontier queue (u16), hash table, scratch
    return cells * (vsz + 4) + ((cells + 1) & ~(size_t)1) * 2 + (size_t)g.block * 12 +
           kScratchWords * 4;
}

BlockedLayout blocked_layout(const Geo& g) {
    BlockedLayout L;
    L.nchunks = (g.words + kChunkWords - 1) / kChunkWords;
    size_t o = 0;
    L.ctrl = o;   o = align256(o + 64);
    L.bctrl = o;  o = align256(o + sizeof(BCtrl));
    L.blk = o;    o = align256(o + L.nchunks * 4);
    L.total = o;
    return L;
}

hipError_t launch_encode_blocked(const Geo& g, const void* x, void* y, uint32_t* b,
                                 hipStream_t s) {
    // Fewer blocks than CUs (large blocks of a sparse gradient): a workgroup
    // per block would leave CUs idle for the whole stream, so the whole chip
    // streams the gradient instead and adds its nonzeros into the zero-filled
    // sketch with global atomics, each batch hashed to its block's rows (the
    // same cells).  Sparse BERT-base (105 blocks of 1024 batches): 0.115 ms
    // per encode with a workgroup per block.
    DeviceInfo di;
    const hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    if (g.nblocks < (uint32_t)di.cus) return launch_encode_dense(g, x, y, b, s);
    if (g.f32) return launch_encode_blocked_t<float>(g, x, y, b, s);
    return launch_encode_blocked_t<int32_t>(g, x, y, b, s);
}

hipError_t launch_decode_blocked(const Geo& g, const void* y_agg, const uint32_t* b_agg,
                                 const DecodeOut& out, const BlockedLayout& L, void* ws,
                                 hipStream_t s) {
    if (g.f32) return launch_decode_blocked_t<float>(g, y_agg, b_agg, out, L, ws, s);
    return launch_decode_blocked_t<int32_t>(g, y_agg, b_agg, out, L, ws, s);
}

}  // namespace hc
