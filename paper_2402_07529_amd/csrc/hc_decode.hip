// hc_decode.hip -- recovery (Algorithm 1, phase II) for gfx950.
//
// Stages (one stream, no host round trips):
//   prep     copy the aggregated sketch into a residual Yw (fp64 for fp32
//            gradients), clear the control block (and, without a plan, the
//            per-cell counters);
//   count    popcount of the bitmap per tile of 16 chunks of 1024 words, and
//            each chunk's offset within its tile;
//   scan     exclusive scan of the tile counts (one workgroup) -> offsets and
//            the support size |S|;
//   support  one wave per chunk: the set bits become the ascending element
//            list E (section 3.2: the index names every nonzero parameter)
//            and, with a plan, every batch's rank offset;
//   counters per cell  cnt = deg * 2^32 + (sum of member positions):  a cell
//            is pure (one live element) exactly when cnt >> 32 == 1, and then
//            its low word is that element's position.  With a plan (the
//            inverse row map of hc_plan.hip) one workgroup per sketch row
//            gathers its counters from the bitmap words of the batches that
//            land on it -- no atomics.  Without a plan every element adds
//            itself to its three cells with 64-bit atomics;
//   round 0  a scan queues the pure cells (round 0's frontier) and, for large
//            sketches, round 0 is peeled, both as ordinary launches over the
//            whole chip; for smaller ones the peel kernel does both itself;
//   peel     one cooperative persistent kernel running the later synchronous
//            rounds (section 3.2, parallel peeling).  The frontier of round r is the
//            list of (cell, element) pairs whose cell became pure during round
//            r-1, kept in one append-only queue.  An element owning several
//            frontier cells is claimed by an atomic OR on its flag byte: the
//            first of its frontier entries to get there recovers
//            x = g_j * Y from its cell (every pure cell of the element holds the
//            same value, exactly so in integer arithmetic), and subtracts g * x
//            and the element from its other two cells with atomics (int32 with
//            a plan: one per cell, the residual riding in the counter word); a
//            cell whose count drops to one joins the next frontier.  Entries whose element
//            is already taken (in this round or an earlier one) do nothing, so
//            the elements peeled in round r are exactly those with a cell in
//            its frontier that were still live when it began.
//            One grid barrier per round (workgroup-scope fences: what a round
//            hands to the next goes through atomics and coherent loads and
//            stores); rounds end when a frontier is empty;
//   leftovers  elements never peeled get the Count Sketch median estimate
//            from the residual sketch (Algorithm 1, last recovery step), on
//            the whole chip: when decoding fails most of the support is left;
//   emit     dense output, recovered mask and COO from E and the values.
#include <type_traits>

#include "hc_device.h"
#include "hc_internal.h"

namespace hc {

namespace {

constexpr int kBlock = 256;
constexpr int kPeelBlock = 1024;  // lanes per workgroup of the persistent peel kernel
constexpr uint32_t kScanCells = 4;  // cells a lane takes per pass of the round-0 scan
constexpr uint32_t kPeelPushCap = 8 * kPeelBlock;  // staged frontier entries per workgroup (64 KiB)
constexpr uint64_t kPeelHalfGridCells = 8ull << 20;  // below this many cells the peel uses half the CUs
constexpr uint64_t kPeelHalfGridCellsInt = 32ull << 20;  // the same with residuals in the counters
constexpr unsigned long long kOne = 1ull << 32;  // one incidence in a packed counter

// The int32 peel can carry a cell's residual in its counter word: value in
// the high 32 bits, deg * 2^k + (sum of member positions) in the low 32, with
// every position below 2^k.  An element leaving the cell subtracts
// (g x) * 2^32 + 2^k + pos: the low part holds the member's own terms, so it
// never borrows from the value, and the value wraps mod 2^32 as the sketch
// does.  One atomic then updates degree, identity and residual together.  It
// needs deg * 2^k + sum < 2^32 in every cell at the start (the low part only
// shrinks); the counter kernels flag any cell where that fails.
__device__ __forceinline__ uint32_t pack_bits(uint64_t nsup) {
    return nsup <= 1 ? 1u : 64u - (uint32_t)__builtin_clzll(nsup - 1);  // nsup <= 2^k
}
__device__ __forceinline__ bool fits_packed(unsigned long long acc, uint32_t k) {
    return ((acc >> 32) << k) + (acc & 0xffffffffull) < (1ull << 32);
}
constexpr uint64_t kChunkBits = (uint64_t)kChunkWords * 32;
constexpr uint64_t kBarrierTimeoutTicks = 500000000ull;  // 5 s at the 100 MHz real-time clock

// Statistics and flags (one 64-byte line; the support scan writes it too).
struct Ctrl {
    unsigned long long n_support;
    unsigned long long recovered;
    unsigned int rounds;
    unsigned int overflow;  // |S| > capacity
    unsigned int abort;     // barrier timeout
    unsigned int done;      // workgroups finished
    unsigned int bad_plan;  // the plan was built for another geometry
    unsigned int nopack;    // some cell's counter does not fit the packed form
    unsigned int pad[6];
};
static_assert(sizeof(Ctrl) == 64, "control block layout");

// Queue and barrier state of the peel.  Every word that many workgroups hit
// in the same few microseconds has a 128-byte line of its own: appends to the
// queue, barrier arrivals and the polls of the waiting workgroups would
// otherwise queue up behind each other on one line (measured on MI355X: a
// barrier of 256 workgroups took about 20 us with the queue length in the
// barrier's line, under 7 us with separate lines).
struct alignas(128) SyncLine {
    unsigned int v[32];
};
struct PeelSync {
    SyncLine tail;    // v[0]: queue length
    SyncLine arrive;  // v[0]: arrivals at the grid barrier, over every barrier of the decode
    SyncLine gen;     // v[0]: barrier generation; v[1]: end of the current frontier
    SyncLine round0;  // v[0]: end of round 0's frontier in the queue
};

// device mirror of hc_decode_info
struct InfoDev {
    unsigned long long n_support, n_recovered, rounds;
    unsigned int success, status;
};

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d);
    return v;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void prep_kernel(const T* __restrict__ y_agg,
                                                      typename Acc<T>::type* __restrict__ yw,
                                                      unsigned long long* __restrict__ cnt,
                                                      uint32_t cells, bool planned,
                                                      Ctrl* __restrict__ ctrl,
                                                      PeelSync* __restrict__ sync,
                                                      uint32_t* __restrict__ mark) {
    if (blockIdx.x == 0) {
        if (threadIdx.x < sizeof(Ctrl) / 4) reinterpret_cast<uint32_t*>(ctrl)[threadIdx.x] = 0u;
        for (uint32_t k = threadIdx.x; k < sizeof(PeelSync) / 4; k += kBlock)
            reinterpret_cast<uint32_t*>(sync)[k] = 0u;
    }
    const uint64_t step = (uint64_t)gridDim.x * kBlock;
    // int32 with a plan: the round-0 scan takes the residual from the
    // aggregate itself (into the counters' high words, or into yw when they
    // do not pack)
    const bool copy = !(std::is_same<T, int32_t>::value && planned);
    for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < cells; i += step) {
        if (copy) yw[i] = (typename Acc<T>::type)y_agg[i];
        if (!planned) cnt[i] = 0ull;
        if (mark != nullptr) mark[i] = 0u;
    }
}

// Bitmap word k, with bits at or past n cleared in the last word.
__device__ __forceinline__ uint32_t load_word(const uint32_t* b, uint64_t k, uint64_t words,
                                              uint32_t last_mask) {
    if (k >= words) return 0u;
    const uint32_t w = b[k];
    return k == words - 1 ? (w & last_mask) : w;
}

// The same for words >= 1, with no branch: past the end it loads the last
// word and returns 0.  A load under a branch is followed, inside the branch,
// by the masking that uses it, so the compiler waits for each such load in
// turn; the row kernels issue theirs together.
__device__ __forceinline__ uint32_t load_word_nb(const uint32_t* b, uint64_t k, uint64_t words,
                                                 uint32_t last_mask) {
    const uint32_t w = b[k < words ? k : words - 1];
    const uint32_t mask = k < words ? (k == words - 1 ? last_mask : 0xffffffffu) : 0u;
    return w & mask;
}

__global__ __launch_bounds__(kBlock) void count_kernel(const uint32_t* __restrict__ b,
                                                       uint64_t words, uint32_t last_mask,
                                                       uint32_t* __restrict__ blk) {
    __shared__ uint32_t s_tmp[kBlock / 64];
    const uint64_t w0 = (uint64_t)blockIdx.x * kChunkWords + 4ull * threadIdx.x;
    uint32_t c = 0;
#pragma unroll
    for (int k = 0; k < 4; k++) c += __popc(load_word(b, w0 + k, words, last_mask));
    c = wave_sum(c);
    if (lane_id() == 0) s_tmp[threadIdx.x >> 6] = c;
    lds_barrier();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int w = 0; w < kBlock / 64; w++) t += s_tmp[w];
        blk[blockIdx.x] = t;
    }
}

// One workgroup of 1024 lanes: chunk counts -> exclusive offsets.  Lane t
// owns a run of consecutive counts whose length is a multiple of 4, read and
// written as 16-byte vectors (the counts start 256-byte aligned).
__device__ __forceinline__ uint4 load_counts4(const uint32_t* blk, uint64_t i, uint64_t nchunks) {
    if (i + 4 <= nchunks) return *reinterpret_cast<const uint4*>(blk + i);
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (i < nchunks) v.x = blk[i];
    if (i + 1 < nchunks) v.y = blk[i + 1];
    if (i + 2 < nchunks) v.z = blk[i + 2];
    return v;
}

__global__ __launch_bounds__(1024) void scan_kernel(uint32_t* __restrict__ blk, uint64_t nchunks,
                                                    Ctrl* __restrict__ ctrl, uint64_t cap) {
    __shared__ uint32_t s_tmp[16];
    const uint64_t per = ((nchunks + 1023) / 1024 + 3) & ~3ull;
    const uint64_t lo = (uint64_t)threadIdx.x * per;
    uint32_t s = 0;
#pragma unroll 8
    for (uint64_t i = lo; i < lo + per; i += 4) {
        const uint4 v = load_counts4(blk, i, nchunks);
        s += v.x + v.y + v.z + v.w;
    }
    uint32_t total;
    uint32_t off = block_exclusive_scan(s, s_tmp, &total);
#pragma unroll 8
    for (uint64_t i = lo; i < lo + per && i < nchunks; i += 4) {
        const uint4 v = load_counts4(blk, i, nchunks);
        uint4 o;
        o.x = off;
        o.y = o.x + v.x;
        o.z = o.y + v.y;
        o.w = o.z + v.z;
        off = o.w + v.w;
        if (i + 4 <= nchunks) {
            *reinterpret_cast<uint4*>(blk + i) = o;
        } else {
            blk[i] = o.x;
            if (i + 1 < nchunks) blk[i + 1] = o.y;
            if (i + 2 < nchunks) blk[i + 2] = o.z;
        }
    }
    if (threadIdx.x == 0) {
        ctrl->n_support = total;
        ctrl->overflow = (uint64_t)total > cap ? 1u : 0u;
    }
}

// ---- support: the element list from the index ------------------------------------
//
// The bitmap is counted in tiles of kTileChunks chunks (one workgroup each,
// 64 KiB: long enough to stream at full rate), writing each tile's count and
// each chunk's offset within its tile; one workgroup scans the tile counts;
// then one wave per chunk writes the chunk offset the emit kernel reads, the
// chunk's run of the ascending element list E (section 3.2: the index names
// every nonzero parameter), cleared peeled flags, and either the
// rank offset of every batch of c parameters (with a plan) or the per-cell
// counters by atomics (without).  A wave per chunk needs no workgroup
// barriers, so a sparse chunk costs little more than its loads, and dense
// bitmaps, whose chunks hold thousands of elements, still spread over the chip.
constexpr uint32_t kTileChunks = 16;

// Words k..k+3 of the bitmap (k a multiple of 4) as load_word reads them; one
// 16-byte load when b is 16-byte aligned and the four lie before the last word.
__device__ __forceinline__ uint4 load_words4(const uint32_t* b, uint64_t k, uint64_t words,
                                             uint32_t last_mask, bool vec) {
    if (vec && k + 4 < words) return *reinterpret_cast<const uint4*>(b + k);
    return make_uint4(load_word(b, k, words, last_mask), load_word(b, k + 1, words, last_mask),
                      load_word(b, k + 2, words, last_mask), load_word(b, k + 3, words, last_mask));
}

__global__ __launch_bounds__(kBlock) void tile_count_kernel(const uint32_t* __restrict__ b,
                                                            uint64_t words, uint32_t last_mask,
                                                            bool vec, uint64_t nchunks,
                                                            uint32_t* __restrict__ cpre,
                                                            uint32_t* __restrict__ tcnt) {
    __shared__ uint32_t s_cnt[kBlock / 64][kTileChunks];
    const uint32_t lane = lane_id();
    const uint32_t wave = threadIdx.x >> 6;
    const uint64_t ch0 = (uint64_t)blockIdx.x * kTileChunks;
    const uint64_t w0 = ch0 * kChunkWords + 4ull * threadIdx.x;
    uint4 v[kTileChunks];
#pragma unroll
    for (uint32_t q = 0; q < kTileChunks; q++)
        v[q] = load_words4(b, w0 + q * kChunkWords, words, last_mask, vec);
#pragma unroll
    for (uint32_t q = 0; q < kTileChunks; q++) {
        const uint32_t c = wave_sum(__popc(v[q].x) + __popc(v[q].y) + __popc(v[q].z) +
                                    __popc(v[q].w));
        if (lane == 0) s_cnt[wave][q] = c;
    }
    lds_barrier();
    if (wave == 0) {
        // lanes 0..kTileChunks-1: chunk counts -> offsets within the tile
        uint32_t c = 0;
        if (lane < kTileChunks)
            for (uint32_t w = 0; w < kBlock / 64; w++) c += s_cnt[w][lane];
        uint32_t x = c;
#pragma unroll
        for (uint32_t d = 1; d < kTileChunks; d <<= 1) {
            const uint32_t y = __shfl_up(x, d);
            if (lane >= d) x += y;
        }
        if (lane < kTileChunks && ch0 + lane < nchunks) cpre[ch0 + lane] = x - c;
        if (lane == kTileChunks - 1) tcnt[blockIdx.x] = x;
    }
}

struct SupportArgs {
    const uint32_t* b;
    const uint32_t* cpre;        // set bits before each chunk within its tile
    const uint32_t* toff;        // set bits before each tile
    uint32_t* blk;               // set bits before each chunk
    uint32_t* woffb;             // with a plan: set bits before each batch (nb + 1 entries)
    uint32_t* elem;
    uint8_t* peeled;             // a byte per element
    unsigned long long* cnt;     // without a plan: counters built by atomics
    Ctrl* ctrl;
    uint64_t words, nchunks, cap, seed;
    uint32_t last_mask, log2wpb, nb, rows, c, cmask, log2c;
    bool vec;  // b is 16-byte aligned
};

// Element pos of E is parameter p: its list entry, its cleared flag and,
// without a plan, its three counter increments.  Positions past the capacity
// are dropped (the decode then reports overflow).
__device__ __forceinline__ void support_put(const SupportArgs& a, uint32_t pos, uint32_t p) {
    if (pos >= a.cap) return;
    a.elem[pos] = p;
    a.peeled[pos] = 0u;
    if (a.woffb == nullptr) {
        const BatchHash h = batch_hash(a.seed, a.rows, a.cmask, p >> a.log2c);
        const uint32_t t = p & a.cmask;
        const unsigned long long inc = kOne + pos;
#pragma unroll
        for (int j = 0; j < 3; j++) atomicAdd(a.cnt + cell_of(h, j, t, a.c, a.cmask), inc);
    }
}

constexpr uint32_t kWaveStage = 1024;  // elements one wave stages in LDS at a time

// The wave stores stage[0, total) as E[base + j], consecutive lanes on
// consecutive elements.  Every lane has written its stage entries.
__device__ __forceinline__ void support_flush(const SupportArgs& a, uint32_t* stage,
                                              uint32_t total, uint32_t base, uint32_t lane) {
    if (total == 0) return;
    // the wave's LDS writes are complete before any lane reads them back
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    for (uint32_t j = lane; j < total; j += 64) support_put(a, base + j, stage[j]);
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();  // the stage is refilled next
}

// One wave, one chunk, in four segments of 256 words; lane l holds words
// 4l..4l+3 of each.  A lane's set bits go to LDS at their rank within the
// segment and the wave then stores the run with consecutive lanes on
// consecutive elements (a lane storing its own run would spread every store
// over 64 lines); a segment with more than kWaveStage elements (over 1/8
// dense) is staged in eight parts.
__global__ __launch_bounds__(kBlock) void support_kernel(SupportArgs a) {
    __shared__ uint32_t s_stage[kBlock / 64][kWaveStage];
    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    const uint64_t chunk = (uint64_t)blockIdx.x * (kBlock / 64) + wave;
    if (chunk >= a.nchunks) return;
    uint32_t* const stage = s_stage[wave];
    const uint64_t c0 = chunk * kChunkWords;
    uint4 v[4];
#pragma unroll
    for (int i = 0; i < 4; i++)
        v[i] = load_words4(a.b, c0 + 256u * i + 4u * lane, a.words, a.last_mask, a.vec);
    uint32_t base = a.toff[chunk / kTileChunks] + a.cpre[chunk];
    if (lane == 0) a.blk[chunk] = base;
    const uint64_t wmask = (1ull << a.log2wpb) - 1ull;
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const uint32_t w4[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
        const uint32_t mine = __popc(w4[0]) + __popc(w4[1]) + __popc(w4[2]) + __popc(w4[3]);
        uint32_t x = mine;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const uint32_t y = __shfl_up(x, d);
            if (lane >= (uint32_t)d) x += y;
        }
        const uint32_t total = __shfl(x, 63);
        uint32_t o = x - mine;  // rank of this lane's first element in the segment
        const uint64_t s0 = c0 + 256u * i;
        const uint64_t w0 = s0 + 4u * lane;
        const bool staged = total <= kWaveStage;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const uint64_t w = w0 + k;
            if (a.woffb != nullptr && w < a.words && (w & wmask) == 0)
                a.woffb[w >> a.log2wpb] = base + o;
            uint32_t bits = staged ? w4[k] : 0u;
            while (bits) {
                stage[o++] = (uint32_t)(w * 32u) + (uint32_t)__builtin_ctz(bits);
                bits &= bits - 1u;
            }
            if (!staged) o += __popc(w4[k]);
        }
        if (staged) {
            support_flush(a, stage, total, base, lane);
        } else {
            // over 1/8 dense: eight passes of 32 words, two lanes per word
            // (16 bits each), at most 1024 elements a pass
            uint32_t pbase = base;
            for (uint32_t part = 0; part < 8; part++) {
                const uint64_t w = s0 + part * 32u + (lane >> 1);
                const uint32_t half = lane & 1u;
                uint32_t bits = (load_word(a.b, w, a.words, a.last_mask) >> (16u * half)) & 0xffffu;
                const uint32_t pc = __popc(bits);
                uint32_t y = pc;
#pragma unroll
                for (int d = 1; d < 64; d <<= 1) {
                    const uint32_t z = __shfl_up(y, d);
                    if (lane >= (uint32_t)d) y += z;
                }
                const uint32_t ptotal = __shfl(y, 63);
                uint32_t q = y - pc;
                while (bits) {
                    stage[q++] = (uint32_t)(w * 32u) + 16u * half + (uint32_t)__builtin_ctz(bits);
                    bits &= bits - 1u;
                }
                support_flush(a, stage, ptotal, pbase, lane);
                pbase += ptotal;
            }
        }
        base += total;
    }
    if (chunk + 1 == a.nchunks && lane == 0 && a.woffb != nullptr) a.woffb[a.nb] = base;
}

// Coherent (agent-scope) 64-bit loads and stores: the peel's grid barrier
// only orders a workgroup's memory operations (it waits for them to complete)
// and does not write back or invalidate the L2, so every value one workgroup
// writes and another reads across a round boundary goes through these (or
// through atomics).
__device__ __forceinline__ unsigned long long ld_agent64(const unsigned long long* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent64(unsigned long long* p, unsigned long long v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---- frontier staging ----------------------------------------------------------

// (cell, element position) pairs whose cell became pure, staged in LDS by one
// workgroup and appended to the global queue with one atomic per flush (a
// single global counter bumped by every wave would serialize the whole grid
// on one cache line).
template <uint32_t CAP>
struct PushBuf {
    static constexpr uint32_t kCap = CAP;
    uint32_t count;
    uint32_t base;
    uint2 item[CAP];
};

template <typename Q>
__device__ __forceinline__ void lds_push(Q& q, bool pred, uint32_t cell, uint32_t pos) {
    const uint64_t m = __ballot(pred);
    if (m == 0) return;
    const uint32_t lane = lane_id();
    const uint32_t leader = (uint32_t)__ffsll((unsigned long long)m) - 1u;
    uint32_t off = 0;
    if (lane == leader) off = atomicAdd(&q.count, (unsigned int)__popcll(m));
    off = __shfl(off, leader);
    if (pred) q.item[off + lanes_below(m)] = make_uint2(cell, pos);
}

// Called by every lane of the workgroup with the same arguments.  Appends the
// staged pairs to the global queue if `force` or if the buffer could not take
// another `room` pushes.  With marks (the fp32 peel), each appended cell's
// mark becomes `markval`: its frontier round plus one.
template <typename Q>
__device__ void flush_pushes(Q& q, bool force, uint32_t room, unsigned int* tail,
                             uint2* queue, uint32_t cells, uint32_t* mark, uint32_t markval) {
    lds_barrier();
    const uint32_t n = q.count;
    lds_barrier();  // every lane has read n before any lane pushes again
    if (n == 0 || (!force && n + room <= Q::kCap)) return;
    if (threadIdx.x == 0) q.base = atomicAdd(tail, n);
    lds_barrier();
    const uint32_t base = q.base;
    for (uint32_t k = threadIdx.x; k < n; k += blockDim.x) {
        if ((uint64_t)base + k >= cells) continue;  // a cell is pushed at most once
        const uint2 it = q.item[k];
        // read by other workgroups after the grid barrier, whose fences do not
        // write back or invalidate the L2: a coherent (agent-scope) store
        st_agent64(reinterpret_cast<unsigned long long*>(queue + base + k),
                   ((unsigned long long)it.y << 32) | it.x);
        if (mark != nullptr)
            __hip_atomic_store(mark + it.x, markval, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    lds_barrier();
    if (threadIdx.x == 0) q.count = 0;
    lds_barrier();
}

// ---- counters by row (planned path) --------------------------------------------

// Called by every lane of a wave: sets ctrl->nopack if some lane's cells do
// not fit the packed form.  One lane of the wave, and only while the flag is
// still clear: a sketch far narrower than its support fails in most cells,
// and an atomic per cell on one word took milliseconds.
__device__ __forceinline__ void flag_unpackable(Ctrl* ctrl, bool fits) {
    if (__ballot(!fits) == 0ull || lane_id() != 0) return;
    if (__hip_atomic_load(&ctrl->nopack, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u)
        atomicOr(&ctrl->nopack, 1u);
}

// Lane l < WPB holds word l of a batch (other lanes hold 0): the set bits in
// words 0..l-1, i.e. the word's rank offset within the batch.
template <uint32_t WPB>
__device__ __forceinline__ uint32_t batch_word_offset(uint32_t word) {
    const uint32_t lane = lane_id();
    const uint32_t pc = __popc(word);
    uint32_t x = pc;
#pragma unroll
    for (uint32_t d = 1; d < WPB; d <<= 1) {
        const uint32_t y = __shfl_up(x, d);
        if (lane >= d) x += y;
    }
    return x - pc;
}

struct CounterArgs {
    const PlanHeader* hdr;
    const uint32_t* rowoff;
    const uint2* entry;
    const uint32_t* b;
    const uint32_t* woffb;  // set bits before each batch (nb + 1 entries)
    unsigned long long* cnt;
    Ctrl* ctrl;
    uint64_t n, seed, words, nb;
    uint32_t rows, c, cmask, cells, last_mask;
};

// One workgroup per sketch row (grid-stride).  Cell k of row r gathers, from
// every (batch b, hash j) in the row's plan entry list, the parameter
// t = (k - bias_j(b)) mod c of batch b: if its bit is set it adds 2^32 + its
// rank in the support.  Integer sums, so the result equals the atomic build
// exactly whatever the order.  Every step issues its global loads together,
// so a row costs a few memory latencies however many batches land on it:
//   screen  each lane takes one plan entry (kBlock at a time) and checks
//           whether any member of the support lies in that batch; the live
//           entries are compacted into an LDS list;
//   stage   the bitmap words and rank offsets of up to kStage live batches
//           are copied into LDS, all lanes loading at once;
//   add     wave w takes staged batches w, w + 4, ...: each lane covers C/64
//           consecutive cells, finds their parameters' bits in the staged
//           words and adds into the row's counters in LDS.
// The row is then written once.  Its pure cells are left for the peel
// kernel's scan: queuing them here took one append on the shared queue tail
// per row (VGG19: 10 K rows, about 0.15 ms of contended atomics).
constexpr uint32_t kStage = 64;  // live batches staged in LDS at a time
constexpr uint64_t kWaveRowsEntries = 8;  // plan entries per row up to which a wave takes a row

template <int C>
__global__ __launch_bounds__(kBlock) void counter_kernel(CounterArgs a) {
    constexpr uint32_t WPB = C / 32;  // bitmap words per batch
    constexpr uint32_t CPL = C / 64;  // cells per lane
    constexpr uint32_t kWaves = kBlock / 64;
    __shared__ unsigned long long s_acc[C];
    __shared__ uint32_t s_word[kStage * WPB];
    __shared__ uint32_t s_boff[kStage];
    __shared__ uint2 s_live[kBlock];
    __shared__ uint32_t s_tmp[kWaves];
    const PlanHeader* hdr = a.hdr;
    const bool ok = hdr->magic == kPlanMagic && hdr->n == a.n && hdr->seed == a.seed &&
                    hdr->c == a.c && hdr->rows == a.rows;
    if (!ok) {
        if (blockIdx.x == 0 && threadIdx.x == 0) a.ctrl->bad_plan = 1u;
        return;
    }
    if (a.ctrl->overflow) return;
    const uint32_t kpack = pack_bits(a.ctrl->n_support);
    const uint32_t lane = lane_id();
    const uint32_t wave = threadIdx.x >> 6;
    for (uint32_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
        for (uint32_t k = threadIdx.x; k < C; k += kBlock) s_acc[k] = 0ull;
        const uint32_t e0 = a.rowoff[row], e1 = a.rowoff[row + 1];
        for (uint32_t base = e0; base < e1; base += kBlock) {
            // screen
            const uint32_t e = base + threadIdx.x;
            uint2 ent = make_uint2(0xffffffffu, 0u);
            bool live = false;
            if (e < e1) {
                ent = a.entry[e];
                if (ent.x < a.nb) live = a.woffb[ent.x + 1] != a.woffb[ent.x];
            }
            uint32_t nlive;
            const uint32_t slot = block_exclusive_scan(live ? 1u : 0u, s_tmp, &nlive);
            if (live) s_live[slot] = ent;
            lds_barrier();
            for (uint32_t g0 = 0; g0 < nlive; g0 += kStage) {
                const uint32_t ng = nlive - g0 < kStage ? nlive - g0 : kStage;
                // stage
                for (uint32_t k = threadIdx.x; k < ng * WPB; k += kBlock) {
                    const uint64_t w = (uint64_t)s_live[g0 + k / WPB].x * WPB + (k % WPB);
                    s_word[k] = load_word(a.b, w, a.words, a.last_mask);
                }
                for (uint32_t k = threadIdx.x; k < ng; k += kBlock)
                    s_boff[k] = a.woffb[s_live[g0 + k].x];
                lds_barrier();
                // add
                for (uint32_t g = wave; g < ng; g += kWaves) {
                    const uint32_t bias = s_live[g0 + g].y & 0xffffu;
                    const uint32_t t0 = (lane * CPL - bias) & (C - 1u);
                    const uint32_t wa = t0 >> 5, wb = ((t0 + CPL - 1u) & (C - 1u)) >> 5;
                    const uint32_t myoff = s_boff[g] + batch_word_offset<WPB>(
                                               lane < WPB ? s_word[g * WPB + lane] : 0u);
                    const uint32_t word_a = s_word[g * WPB + wa], off_a = __shfl(myoff, wa);
                    const uint32_t word_b = s_word[g * WPB + wb], off_b = __shfl(myoff, wb);
#pragma unroll
                    for (uint32_t i = 0; i < CPL; i++) {
                        const uint32_t t = (t0 + i) & (C - 1u);
                        const bool first = (t >> 5) == wa;
                        const uint32_t word = first ? word_a : word_b;
                        const uint32_t bit = t & 31u;
                        if ((word >> bit) & 1u) {
                            const uint32_t rank = (first ? off_a : off_b) +
                                                  __popc(word & ((1u << bit) - 1u));
                            atomicAdd(&s_acc[lane * CPL + i], kOne + rank);
                        }
                    }
                }
                lds_barrier();  // the staging buffers are reused
            }
        }
        bool fits = true;
        for (uint32_t k = threadIdx.x; k < C; k += kBlock) {
            const unsigned long long acc = s_acc[k];
            a.cnt[row * C + k] = acc;
            fits = fits && fits_packed(acc, kpack);
        }
        flag_unpackable(a.ctrl, fits);
        lds_barrier();  // s_acc is cleared for the next row
    }
}

// Rows that few batches land on (a sketch much wider than the support): one
// wave per row, no workgroup barriers.  Lane e screens entry e of the row; the
// live batches are visited in turn: lanes 0..C/32-1 load the batch's bitmap
// words and rank offsets, every lane takes the (at most two) words covering
// its C/64 consecutive cells by shuffle and adds into its own cells of the
// wave's copy of the row in LDS.  The row is written with plain stores.
template <int C>
__global__ __launch_bounds__(kBlock) void counter_wave_kernel(CounterArgs a) {
    constexpr uint32_t WPB = C / 32;  // bitmap words per batch
    constexpr uint32_t CPL = C / 64;  // cells per lane
    constexpr uint32_t kWaves = kBlock / 64;
    __shared__ unsigned long long s_acc[kWaves * C];
    const PlanHeader* hdr = a.hdr;
    const bool ok = hdr->magic == kPlanMagic && hdr->n == a.n && hdr->seed == a.seed &&
                    hdr->c == a.c && hdr->rows == a.rows;
    if (!ok) {
        if (blockIdx.x == 0 && threadIdx.x == 0) a.ctrl->bad_plan = 1u;
        return;
    }
    if (a.ctrl->overflow) return;
    const uint32_t kpack = pack_bits(a.ctrl->n_support);
    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    unsigned long long* const acc = s_acc + wave * C;
    const uint32_t nwaves = gridDim.x * kWaves;
    for (uint32_t row = blockIdx.x * kWaves + wave; row < a.rows; row += nwaves) {
#pragma unroll
        for (uint32_t i = 0; i < CPL; i++) acc[lane * CPL + i] = 0ull;
        const uint32_t e0 = a.rowoff[row], e1 = a.rowoff[row + 1];
        for (uint32_t base = e0; base < e1; base += 64u) {
            const uint32_t e = base + lane;
            uint2 ent = make_uint2(0xffffffffu, 0u);
            bool live = false;
            if (e < e1) {
                ent = a.entry[e];
                if (ent.x < a.nb) live = a.woffb[ent.x + 1] != a.woffb[ent.x];
            }
            uint64_t m = __ballot(live);
            while (m) {
                const uint32_t src = (uint32_t)__ffsll((unsigned long long)m) - 1u;
                m &= m - 1ull;
                const uint32_t bidx = __shfl(ent.x, src);
                const uint32_t bias = __shfl(ent.y, src) & 0xffffu;
                const uint64_t ws = (uint64_t)bidx * WPB;
                const uint32_t boff = a.woffb[bidx];
                const uint32_t myword = lane < WPB ? load_word(a.b, ws + lane, a.words, a.last_mask) : 0u;
                const uint32_t myoff = boff + batch_word_offset<WPB>(myword);
                const uint32_t t0 = (lane * CPL - bias) & (C - 1u);
                const uint32_t wa = t0 >> 5, wb = ((t0 + CPL - 1u) & (C - 1u)) >> 5;
                const uint32_t word_a = __shfl(myword, wa), off_a = __shfl(myoff, wa);
                const uint32_t word_b = __shfl(myword, wb), off_b = __shfl(myoff, wb);
#pragma unroll
                for (uint32_t i = 0; i < CPL; i++) {
                    const uint32_t t = (t0 + i) & (C - 1u);
                    const bool first = (t >> 5) == wa;
                    const uint32_t word = first ? word_a : word_b;
                    const uint32_t bit = t & 31u;
                    if ((word >> bit) & 1u) {
                        const uint32_t rank = (first ? off_a : off_b) +
                                              __popc(word & ((1u << bit) - 1u));
                        acc[lane * CPL + i] += kOne + rank;
                    }
                }
            }
        }
        unsigned long long* dst = a.cnt + (uint64_t)row * C;
        bool fits = true;
#pragma unroll
        for (uint32_t i = 0; i < CPL; i++) {
            const unsigned long long v = acc[i * 64u + lane];
            dst[i * 64u + lane] = v;
            fits = fits && fits_packed(v, kpack);
        }
        flag_unpackable(a.ctrl, fits);
    }
}

// The live batches of one screened chunk (lanes with `live`, their batch,
// rotation and rank offset in bidx, bias and boff) added into the wave's row
// of counters acc: kGroup batches per wave-wide load (WPB lanes each, one
// bitmap word per lane), kUnroll loads in flight together; each lane turns
// its word's set bits into cells and ranks.
template <int C>
__device__ __forceinline__ void add_live_batches(const CounterArgs& a, bool live, uint32_t bidx,
                                                 uint32_t bias, uint32_t boff,
                                                 unsigned long long* acc) {
    constexpr uint32_t WPB = C / 32;       // bitmap words per batch
    constexpr uint32_t kGroup = 64 / WPB;  // batches per wave-wide load
    constexpr uint32_t kUnroll = 4;        // wave-wide loads in flight
    const uint32_t lane = lane_id();
    const uint32_t seg = lane / WPB;  // which batch of a group this lane serves
    const uint32_t wl = lane % WPB;   // which word of it
    uint64_t m = __ballot(live);
    while (m != 0ull) {
        uint32_t word[kUnroll], gbias[kUnroll], goff[kUnroll];
        bool have[kUnroll];
#pragma unroll
        for (uint32_t u = 0; u < kUnroll; u++) {
            // this segment's batch: the seg-th live lane left, if any
            uint64_t mm = m;
#pragma unroll
            for (uint32_t q = 0; q < kGroup; q++)
                if (q < seg && mm != 0ull) mm &= mm - 1ull;
            have[u] = mm != 0ull;
            const uint32_t src = have[u] ? (uint32_t)__ffsll((unsigned long long)mm) - 1u : 0u;
            const uint32_t gb = (uint32_t)__shfl(bidx, (int)src);
            gbias[u] = (uint32_t)__shfl(bias, (int)src);
            goff[u] = (uint32_t)__shfl(boff, (int)src);
            // loaded whether or not the segment has a batch (gb is then some
            // lane's entry, possibly none: the load is clamped), and dropped
            // below, so that no load sits under a branch
            word[u] = load_word_nb(a.b, (uint64_t)gb * WPB + wl, a.words, a.last_mask);
#pragma unroll
            for (uint32_t q = 0; q < kGroup; q++)  // the group's batches are taken
                if (m != 0ull) m &= m - 1ull;
        }
#pragma unroll
        for (uint32_t u = 0; u < kUnroll; u++) {
            if (!have[u]) word[u] = 0u;
            // rank of the word's first bit: the batch's offset plus the
            // popcounts of its earlier words (a scan within the segment)
            const uint32_t pc = __popc(word[u]);
            uint32_t x = pc;
#pragma unroll
            for (uint32_t d = 1; d < WPB; d <<= 1) {
                const uint32_t y = __shfl_up(x, d);
                if (wl >= d) x += y;
            }
            uint32_t rank = goff[u] + x - pc;
            uint32_t w = have[u] ? word[u] : 0u;
            while (w != 0u) {
                const uint32_t bit = (uint32_t)__builtin_ctz(w);
                w &= w - 1u;
                atomicAdd(&acc[(32u * wl + bit + gbias[u]) & (uint32_t)(C - 1)], kOne + rank);
                rank++;
            }
        }
    }
}

constexpr uint32_t kScreen = 4;  // chunks of 64 plan entries a row wave screens together

// Screens kScreen chunks of 64 plan entries of a row, from entry cs (< e1):
// a lane per entry, is any member of the support in the entry's batch?  Gives
// each entry's batch (0xffffffff: none), its packed hash word, the batch's
// rank offset and whether it is live.  Every load is issued unconditionally,
// at a clamped index, so that the entries' loads are in flight together and
// then the rank offsets'.
__device__ __forceinline__ void screen_entries(const CounterArgs& a, uint32_t cs, uint32_t e1,
                                               uint32_t (&bidx)[kScreen], uint32_t (&ey)[kScreen],
                                               uint32_t (&boff)[kScreen], bool (&live)[kScreen]) {
    const uint32_t lane = lane_id();
    uint2 ent[kScreen];
#pragma unroll
    for (uint32_t h = 0; h < kScreen; h++) {
        const uint32_t e = cs + 64u * h + lane;
        ent[h] = a.entry[e < e1 ? e : e1 - 1u];
    }
    uint32_t lo[kScreen], hi[kScreen];
#pragma unroll
    for (uint32_t h = 0; h < kScreen; h++) {
        const bool ok = cs + 64u * h + lane < e1 && ent[h].x < a.nb;
        bidx[h] = ok ? ent[h].x : 0xffffffffu;
        const uint32_t bi = ok ? ent[h].x : 0u;
        lo[h] = a.woffb[bi];
        hi[h] = a.woffb[bi + 1];
    }
#pragma unroll
    for (uint32_t h = 0; h < kScreen; h++) {
        ey[h] = ent[h].y;
        boff[h] = lo[h];
        live[h] = bidx[h] != 0xffffffffu && hi[h] != lo[h];
    }
}

// Row `row`'s counters, built by one wave in its LDS (acc): the wave screens
// kScreen chunks of 64 plan entries with their loads in flight (a lane per
// entry: is any member of the support in the batch?), then adds the live
// batches' members bit by bit (add_live_batches).
template <int C>
__device__ void build_row(const CounterArgs& a, uint32_t row, unsigned long long* acc) {
    const uint32_t lane = lane_id();
    // a wave's LDS operations complete in order: the previous row's reads are
    // done before these stores
    for (uint32_t k = lane; k < (uint32_t)C; k += 64) acc[k] = 0ull;
    const uint32_t e0 = a.rowoff[row], e1 = a.rowoff[row + 1];
    for (uint32_t cs = e0; cs < e1; cs += 64u * kScreen) {
        uint32_t bidx[kScreen], ey[kScreen], boff[kScreen];
        bool live[kScreen];
        screen_entries(a, cs, e1, bidx, ey, boff, live);
#pragma unroll
        for (uint32_t h = 0; h < kScreen; h++)
            add_live_batches<C>(a, live[h], bidx[h], ey[h] & 0xffffu, boff[h], acc);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // every lane's LDS adds have landed
    __builtin_amdgcn_wave_barrier();
}

// Whether the plan was built for this geometry; if not, flags it (the decode
// then reports status 3).
__device__ __forceinline__ bool plan_matches(const CounterArgs& a) {
    const PlanHeader* hdr = a.hdr;
    const bool ok = hdr->magic == kPlanMagic && hdr->n == a.n && hdr->seed == a.seed &&
                    hdr->c == a.c && hdr->rows == a.rows;
    if (!ok && blockIdx.x == 0 && threadIdx.x == 0) a.ctrl->bad_plan = 1u;
    return ok;
}

// One wave per sketch row (grid-stride), its counters in the wave's LDS: the
// same counters as counter_kernel, for sketches with rows to spare.  The row
// is written once.  A wave per row needs no workgroup barriers and keeps four
// times as many rows in flight as a workgroup per row (VGG19: 10 K rows, the
// counters went from 178 to 101 us); with few long rows (NCF: 1.9 K rows of
// 1.7 K entries, a few dense words per batch) it left SIMDs idle and ran
// twice as long as counter_kernel.
template <int C>
__global__ __launch_bounds__(kBlock) void counter_rows_kernel(CounterArgs a) {
    constexpr uint32_t kWaves = kBlock / 64;
    __shared__ unsigned long long s_acc[kWaves * C];
    if (!plan_matches(a)) return;
    if (a.ctrl->overflow) return;
    const uint32_t kpack = pack_bits(a.ctrl->n_support);
    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    unsigned long long* const acc = s_acc + wave * C;
    const uint32_t nwaves = gridDim.x * kWaves;
    for (uint32_t row = blockIdx.x * kWaves + wave; row < a.rows; row += nwaves) {
        build_row<C>(a, row, acc);
        unsigned long long* dst = a.cnt + (uint64_t)row * C;
        bool fits = true;
        for (uint32_t k = lane; k < (uint32_t)C; k += 64) {
            const unsigned long long v = acc[k];
            dst[k] = v;
            fits = fits && fits_packed(v, kpack);
        }
        flag_unpackable(a.ctrl, fits);
    }
}

// ---- round 0 by rows (int32 with a plan, rows to spare) --------------------------
//
// Round 0 of the peel (Algorithm 1) recovers every element that has a pure
// cell: x = g Y at that cell, exact in int32.  Taken entry by entry, each of
// those elements costs its two other cells a scattered 64-bit atomic, which
// bounds the round at the chip's scattered-atomic rate (VGG19: 2.2 M
// elements, 0.3 ms).  Here round 0 is two passes over the rows through the
// plan instead, every update landing in the row's counters in LDS:
//   pure_rows    builds each row's counters as counter_rows_kernel does and,
//                for each pure cell, writes its element's value and sets its
//                flag (an element with several pure cells gets the same
//                value from each);
//   round0_rows  builds each row's counters again without the flagged
//                elements, subtracts their values from the residual, writes
//                the counters the peel kernel continues from (packed with the
//                residuals, or counters and residuals apart) and queues the
//                cells left pure: round 1's frontier.
// The round's elements, values and counters are those of the entry-by-entry
// round; only the order of round 1's frontier in the queue differs.
struct Round0Args {
    CounterArgs c;
    const int32_t* y_agg;
    int32_t* vals;
    uint8_t* peeled;
    const uint32_t* elem;
    int32_t* yw;
    uint2* queue;
    unsigned int* tail;
    uint32_t log2c;
};

template <int C>
__global__ __launch_bounds__(kBlock) void pure_rows_kernel(Round0Args r) {
    constexpr uint32_t kWaves = kBlock / 64;
    constexpr uint32_t CPL = C / 64;  // cells per lane
    __shared__ unsigned long long s_acc[kWaves * C];
    const CounterArgs& a = r.c;
    if (!plan_matches(a)) return;
    if (a.ctrl->overflow) return;
    const uint32_t nsup = (uint32_t)a.ctrl->n_support;
    const uint32_t kpack = pack_bits(nsup);
    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    unsigned long long* const acc = s_acc + wave * C;
    const uint32_t nwaves = gridDim.x * kWaves;
    for (uint32_t row = blockIdx.x * kWaves + wave; row < a.rows; row += nwaves) {
        build_row<C>(a, row, acc);
        bool fits = true;
        bool pure[CPL];
        uint32_t pos[CPL], p[CPL];
        int32_t y[CPL];
        // the pure cells' elements and sketch values, their loads in flight together
#pragma unroll
        for (uint32_t i = 0; i < CPL; i++) {
            const unsigned long long v = acc[lane + 64u * i];
            fits = fits && fits_packed(v, kpack);
            pos[i] = (uint32_t)v;
            pure[i] = (v >> 32) == 1ull && pos[i] < nsup;
            p[i] = r.elem[pure[i] ? pos[i] : 0u];
            y[i] = r.y_agg[(uint64_t)row * C + lane + 64u * i];
        }
        flag_unpackable(a.ctrl, fits);
#pragma unroll
        for (uint32_t i = 0; i < CPL; i++) {
            if (!pure[i]) continue;
            // the element's hash that lands in this row (its three rows differ)
            const BatchHash h = batch_hash(a.seed, a.rows, a.cmask, p[i] >> r.log2c);
            const uint32_t j = h.row[0] == row ? 0u : (h.row[1] == row ? 1u : 2u);
            r.vals[pos[i]] = Val<int32_t>::sign(y[i], (h.neg >> j) & 1u);
            r.peeled[pos[i]] = 1u;
        }
    }
}

// Like add_live_batches, for round0_rows.  PHASE 0: packed counters (the
// residual in the high word, deg * 2^kp + sum of positions in the low), the
// flagged members' -g x added to the residual and the others counted;
// PHASE 1: unpacked counters (deg * 2^32 + sum of positions) of the members
// not flagged; PHASE 2: the flagged members' -g x in the low word.  The flags
// and values of each batch's first kWin members (ranks are consecutive within
// a batch) are loaded with the bitmap words, by the batch's WPB lanes, and
// staged in the wave's window in LDS (win: kR0Unroll * 64 / WPB batches of
// kWin values, then as many of kWin flag bytes); members past that read
// memory.  Counts into e0 the flagged members met through their hash j = 0:
// each element once.
// wave-wide bitmap loads in flight per round0_rows wave: with two, the larger
// LDS window left three workgroups per CU instead of four, and VGG19's pass
// took 20 us longer
constexpr uint32_t kR0Unroll = 1;

template <int C, int PHASE>
__device__ __forceinline__ void sub_live_batches(const Round0Args& r, bool live, uint32_t bidx,
                                                 uint32_t ey, uint32_t boff,
                                                 unsigned long long* acc, uint32_t* win,
                                                 uint32_t kp, uint32_t nsup, uint32_t& e0) {
    constexpr uint32_t WPB = C / 32;       // bitmap words per batch
    constexpr uint32_t kGroup = 64 / WPB;  // batches per wave-wide load
    constexpr uint32_t kWin = 4 * WPB;     // members per batch staged in the window
    constexpr uint32_t kWinVals = kR0Unroll * kGroup * kWin;  // = 4 * 64 * kR0Unroll
    const CounterArgs& a = r.c;
    const uint32_t lane = lane_id();
    const uint32_t seg = lane / WPB;
    const uint32_t wl = lane % WPB;
    uint8_t* const wflag = reinterpret_cast<uint8_t*>(win + kWinVals);
    uint64_t m = __ballot(live);
    while (m != 0ull) {
        uint32_t word[kR0Unroll], gy[kR0Unroll], goff[kR0Unroll], fw[kR0Unroll],
            vw[kR0Unroll][4];
        bool have[kR0Unroll];
#pragma unroll
        for (uint32_t u = 0; u < kR0Unroll; u++) {
            uint64_t mm = m;
#pragma unroll
            for (uint32_t q = 0; q < kGroup; q++)
                if (q < seg && mm != 0ull) mm &= mm - 1ull;
            have[u] = mm != 0ull;
            const uint32_t src = have[u] ? (uint32_t)__ffsll((unsigned long long)mm) - 1u : 0u;
            const uint32_t gb = (uint32_t)__shfl(bidx, (int)src);
            gy[u] = (uint32_t)__shfl(ey, (int)src);
            goff[u] = (uint32_t)__shfl(boff, (int)src);
            // every load unconditional, at a clamped index, and dropped below
            // where it is not wanted (see add_live_batches)
            word[u] = load_word_nb(a.b, (uint64_t)gb * WPB + wl, a.words, a.last_mask);
            // flag bytes [fb, fb + 4) and values [vb, vb + 4) of the batch's
            // first kWin members (the arrays hold at least 256 bytes)
            const uint32_t fb = (goff[u] & ~3u) + 4u * wl;
            fw[u] = *reinterpret_cast<const uint32_t*>(r.peeled + (fb < nsup ? fb : 0u));
            if (!(have[u] && fb < nsup)) fw[u] = 0u;
#pragma unroll
            for (uint32_t i = 0; i < 4; i++) {
                const uint32_t vb = goff[u] + 4u * wl + i;
                vw[u][i] = PHASE != 1 ? (uint32_t)r.vals[vb < nsup ? vb : 0u] : 0u;
            }
#pragma unroll
            for (uint32_t q = 0; q < kGroup; q++)
                if (m != 0ull) m &= m - 1ull;
        }
        // the window: the previous batches' reads were issued before these
        // stores, and a wave's LDS operations complete in order
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
#pragma unroll
        for (uint32_t u = 0; u < kR0Unroll; u++) {
            const uint32_t wb = (u * kGroup + seg) * kWin + 4u * wl;
            *reinterpret_cast<uint32_t*>(wflag + wb) = fw[u];
            if (PHASE != 1) {
#pragma unroll
                for (uint32_t i = 0; i < 4; i++) win[wb + i] = vw[u][i];
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (uint32_t u = 0; u < kR0Unroll; u++) {
            if (!have[u]) word[u] = 0u;
            const uint32_t pc = __popc(word[u]);
            uint32_t x = pc;
#pragma unroll
            for (uint32_t d = 1; d < WPB; d <<= 1) {
                const uint32_t y = __shfl_up(x, d);
                if (wl >= d) x += y;
            }
            uint32_t rank = goff[u] + x - pc;
            const uint32_t bias = gy[u] & 0xffffu;
            const uint32_t j = (gy[u] >> 16) & 3u;
            const bool neg = (gy[u] >> 31) != 0u;
            const uint32_t fbase = goff[u] & ~3u;
            const uint32_t wbase = (u * kGroup + seg) * kWin;
            uint32_t w = have[u] ? word[u] : 0u;
            while (w != 0u) {
                const uint32_t bit = (uint32_t)__builtin_ctz(w);
                w &= w - 1u;
                const uint32_t fi = rank - fbase, vi = rank - goff[u];
                const bool fl = (fi < kWin ? wflag[wbase + fi] : r.peeled[rank]) != 0u;
                const uint32_t cell = (32u * wl + bit + bias) & (uint32_t)(C - 1);
                if (PHASE == 1) {
                    if (!fl) atomicAdd(&acc[cell], kOne + rank);
                } else if (fl) {
                    const uint32_t xv = vi < kWin ? win[wbase + vi] : (uint32_t)r.vals[rank];
                    const uint32_t gx = neg ? xv : 0u - xv;  // -g x
                    atomicAdd(&acc[cell], PHASE == 0 ? (unsigned long long)gx << 32
                                                     : (unsigned long long)gx);
                } else if (PHASE == 0) {
                    atomicAdd(&acc[cell], (1ull << kp) + rank);
                }
                if (PHASE != 2 && fl && j == 0u) e0++;
                rank++;
            }
        }
    }
}

template <int C, int PHASE>
__device__ void round0_row(const Round0Args& r, uint32_t row, unsigned long long* acc,
                           uint32_t* win, uint32_t kp, uint32_t nsup, uint32_t& e0) {
    const CounterArgs& a = r.c;
    const uint32_t lane = lane_id();
    // a wave's LDS operations complete in order: the previous row's reads are
    // done before these stores
    constexpr uint32_t CPL = C / 64;
    uint32_t y[CPL];
#pragma unroll
    for (uint32_t i = 0; i < CPL; i++)
        y[i] = PHASE == 1 ? 0u : (uint32_t)r.y_agg[(uint64_t)row * C + lane + 64u * i];
#pragma unroll
    for (uint32_t i = 0; i < CPL; i++)
        acc[lane + 64u * i] = PHASE == 0 ? (unsigned long long)y[i] << 32 : (unsigned long long)y[i];
    const uint32_t r0 = a.rowoff[row], r1 = a.rowoff[row + 1];
    for (uint32_t cs = r0; cs < r1; cs += 64u * kScreen) {
        uint32_t bidx[kScreen], ey[kScreen], boff[kScreen];
        bool live[kScreen];
        screen_entries(a, cs, r1, bidx, ey, boff, live);
#pragma unroll
        for (uint32_t h = 0; h < kScreen; h++)
            sub_live_batches<C, PHASE>(r, live[h], bidx[h], ey[h], boff[h], acc, win, kp, nsup,
                                       e0);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // every lane's LDS adds have landed
    __builtin_amdgcn_wave_barrier();
}

// Writes the row's counters (cnt) and queues its pure cells with their
// elements (packed: positions in the low kp bits; unpacked: the low word).
template <int C>
__device__ void round0_write_row(const Round0Args& r, uint32_t row,
                                 const unsigned long long* acc, bool packed, uint32_t kp) {
    constexpr uint32_t CPL = C / 64;
    const CounterArgs& a = r.c;
    const uint32_t lane = lane_id();
    uint32_t npush = 0, mine = 0;  // bit i of mine: cell lane + 64 i is pure
    unsigned long long* dst = a.cnt + (uint64_t)row * C;
#pragma unroll
    for (uint32_t i = 0; i < CPL; i++) {
        const unsigned long long v = acc[lane + 64u * i];
        dst[lane + 64u * i] = v;
        const bool pure = packed ? ((uint32_t)v >> kp) == 1u : (v >> 32) == 1ull;
        mine |= (uint32_t)pure << i;
        npush += (uint32_t)__popcll(__ballot(pure));
    }
    if (npush == 0u) return;
    uint32_t base = 0;
    if (lane == 0) base = atomicAdd(r.tail, npush);
    base = (uint32_t)__shfl((int)base, 0);
#pragma unroll
    for (uint32_t i = 0; i < CPL; i++) {
        const bool pure = (mine >> i) & 1u;
        const uint64_t bal = __ballot(pure);
        if (pure) {
            const uint64_t slot = (uint64_t)base + lanes_below(bal);
            const unsigned long long v = acc[lane + 64u * i];
            const uint32_t pos = packed ? (uint32_t)v & ((1u << kp) - 1u) : (uint32_t)v;
            if (slot < a.cells)  // a cell is queued at most once
                r.queue[slot] = make_uint2(row * (uint32_t)C + lane + 64u * i, pos);
        }
        base += (uint32_t)__popcll(bal);
    }
}

template <int C>
__global__ __launch_bounds__(kBlock) void round0_rows_kernel(Round0Args r) {
    constexpr uint32_t kWaves = kBlock / 64;
    // per wave: the row's counters, and the window of kR0Unroll * 64 * 4
    // values and as many flag bytes (sub_live_batches)
    constexpr uint32_t kWinWords = kR0Unroll * 64 * 4 + kR0Unroll * 64;
    __shared__ unsigned long long s_acc[kWaves * C];
    __shared__ uint32_t s_win[kWaves * kWinWords];
    __shared__ uint32_t s_red;
    const CounterArgs& a = r.c;
    Ctrl* ctrl = a.ctrl;
    if (ctrl->overflow != 0 || ctrl->bad_plan != 0) return;
    if (threadIdx.x == 0) s_red = 0;
    lds_barrier();
    const uint32_t nsup = (uint32_t)ctrl->n_support;
    const uint32_t kp = pack_bits(nsup);
    const bool packed = ctrl->nopack == 0;
    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    unsigned long long* const acc = s_acc + wave * C;
    uint32_t* const win = s_win + wave * kWinWords;
    const uint32_t nwaves = gridDim.x * kWaves;
    uint32_t e0 = 0;
    for (uint32_t row = blockIdx.x * kWaves + wave; row < a.rows; row += nwaves) {
        if (packed) {
            round0_row<C, 0>(r, row, acc, win, kp, nsup, e0);
            round0_write_row<C>(r, row, acc, true, kp);
        } else {
            round0_row<C, 1>(r, row, acc, win, kp, nsup, e0);
            round0_write_row<C>(r, row, acc, false, kp);
            round0_row<C, 2>(r, row, acc, win, kp, nsup, e0);
            for (uint32_t k = lane; k < (uint32_t)C; k += 64)
                r.yw[(uint64_t)row * C + k] = (int32_t)(uint32_t)acc[k];
        }
    }
    e0 = wave_sum(e0);
    if (lane == 0 && e0 != 0u) atomicAdd(&s_red, e0);
    lds_barrier();
    if (threadIdx.x == 0 && s_red != 0u) {
        atomicAdd(&ctrl->recovered, (unsigned long long)s_red);
        atomicMax(&ctrl->rounds, 1u);  // recoveries in round 0
    }
}

// ---- peel ------------------------------------------------------------------------

template <typename T>
struct PeelArgs {  // T: the decode-side arithmetic type
    Ctrl* ctrl;
    PeelSync* sync;
    const uint32_t* elem;
    T* vals;
    uint8_t* peeled;  // a byte per element, set and tested through its 32-bit word
    unsigned long long* cnt;
    T* yw;
    const int32_t* y_agg;  // int32: the aggregated sketch (the residual before round 0)
    uint2* queue;
    uint32_t* mark;  // fp32 peel: per cell, its frontier round + 1 (0: never queued)
    InfoDev* info;
    uint64_t seed;
    uint32_t rows, c, cmask, log2c, cells;
    bool counted;   // a counter kernel built the counters (and checked their packing)
    bool split0;    // round 0 ran before the peel kernel, as whole-chip launches
};

// Round-0 scan of an int32 sketch with a plan: the residual starts as the
// aggregate, in the counter's high word when packed (v: the counter as the
// counter kernel built it), else in yw.
template <typename T>
__device__ __forceinline__ void scan_residual(const PeelArgs<T>& a, uint64_t cidx,
                                              unsigned long long v, bool packed, uint32_t kp) {
    if constexpr (std::is_same<T, int32_t>::value) {
        if (!a.counted || cidx >= a.cells) return;
        const uint32_t y = (uint32_t)a.y_agg[cidx];
        if (packed)
            st_agent64(a.cnt + cidx,
                       ((unsigned long long)y << 32) | (((v >> 32) << kp) + (v & 0xffffffffull)));
        else
            __hip_atomic_store(a.yw + cidx, (int32_t)y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// One frontier entry (cell cidx, element position pos), for the kernel below.
// PACKED: int32 residuals ride in the counter words (kp position bits).
// Sets the (at most two) cells that became pure, with their elements.
// Integer peels (T = int32): the first frontier entry of an element to claim
// its flag recovers it; any of its pure cells holds the same value exactly.
// The fp32 gradient's peel (T = double, with marks): every element is
// recovered from the pure cell with the smallest j among those in the round's
// frontier, as the synchronous rounds define it.  In floating point the pure
// cells of an element carry different rounding, so this makes the result
// independent of the order in which entries are taken.  A cell of a live
// element that is in the frontier holds that element alone, and a live
// element's cells enter the frontier only in the round before it is
// recovered, so "mark == r + 1" tells exactly which of its cells are pure at
// the start of round r; the element's entries with a larger j stand aside and
// no claim is needed.  Its flag, set with a plain store, stops entries of
// later rounds (a cell of the element that became pure while it was being
// recovered).
template <typename T, bool PACKED>
__device__ __forceinline__ void peel_entry(const PeelArgs<T>& a, uint32_t cidx, uint32_t pos,
                                           uint32_t kp, uint32_t r, uint32_t& recovered,
                                           uint32_t& last_round, bool (&push)[2],
                                           uint32_t (&pcell)[2], uint32_t (&ppos)[2]) {
    constexpr bool kMarks = std::is_same<T, double>::value;
    // the element's flag byte within its 32-bit word (the flags are 256-byte
    // aligned): a byte rather than a word per element keeps the flags a
    // quarter of the size in the caches; claims of four neighbouring
    // elements share a word but rarely meet in time
    unsigned int* const fword = reinterpret_cast<unsigned int*>(a.peeled + (pos & ~3u));
    const uint32_t fbit = 1u << (8u * (pos & 3u));
    // the cell's residual first: a frontier cell holds one element, so no
    // other entry changes it this round (and with this load ahead of the
    // claim the two versions of this function share no leading code, which
    // the compiler had hoisted above their differing loads)
    unsigned long long wcell = 0;
    T ycell = T(0);
    if (PACKED) wcell = ld_agent64(a.cnt + cidx);
    else ycell = __hip_atomic_load(a.yw + cidx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bool taken;
    if (kMarks)
        taken = (__hip_atomic_load(fword, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & fbit) != 0u;
    else
        taken = (atomicOr(fword, fbit) & fbit) != 0u;
    const uint32_t p = a.elem[pos];
    const BatchHash h = batch_hash(a.seed, a.rows, a.cmask, p >> a.log2c);
    const uint32_t t = p & a.cmask;
    uint32_t cl[3];
#pragma unroll
    for (int j = 0; j < 3; j++) cl[j] = cell_of(h, j, t, a.c, a.cmask);
    const int j = cl[0] == cidx ? 0 : (cl[1] == cidx ? 1 : 2);
    // the cell's load stays beside the claim's and the element's: otherwise
    // the compiler sinks it past the test below, a memory latency later
    if (PACKED) {
        const uint32_t hi = (uint32_t)(wcell >> 32);
        asm volatile("" : : "v"(hi));
    } else {
        asm volatile("" : : "v"(ycell));
    }
    if (taken || cl[j] != cidx) return;
    if (kMarks) {
        for (int jj = 0; jj < j; jj++)
            if (__hip_atomic_load(a.mark + cl[jj], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                r + 1u)
                return;
        atomicOr(fword, fbit);  // neighbours' flags share the word
    }
    if (PACKED) ycell = (T)(int32_t)(uint32_t)(wcell >> 32);
    const T val = Val<T>::sign(ycell, (h.neg >> j) & 1u);
    a.vals[pos] = val;
    recovered++;
    last_round = r + 1u;
    const int jo[2] = {j == 0 ? 1 : 0, j == 2 ? 1 : 2};
    unsigned long long old[2], inc[2];
#pragma unroll
    for (int u = 0; u < 2; u++) {
        const T gx = Val<T>::sign(val, !((h.neg >> jo[u]) & 1u));  // -g * x
        if (PACKED)
            inc[u] = ((unsigned long long)(uint32_t)(int32_t)gx << 32) - ((1ull << kp) + pos);
        else
            inc[u] = 0ull - (kOne + pos);
        old[u] = atomicAdd(a.cnt + cl[jo[u]], inc[u]);
        if (!PACKED) Val<T>::atomic_add(a.yw + cl[jo[u]], gx);
    }
#pragma unroll
    for (int u = 0; u < 2; u++) {
        const unsigned long long nw = old[u] + inc[u];
        pcell[u] = cl[jo[u]];
        if (PACKED) {
            const uint32_t low = (uint32_t)nw;
            push[u] = (low >> kp) == 1u;
            ppos[u] = low & ((1u << kp) - 1u);
        } else {
            push[u] = (nw >> 32) == 1ull;
            ppos[u] = (uint32_t)nw;
        }
    }
}

// Grid-wide barrier in two levels: the workgroups of group g (blockIdx % G)
// arrive on the group's counter, the last of each group on the top counter,
// and the last of those publishes the end of the next frontier and bumps the
// generation that everyone polls.  Each workgroup makes its writes visible
// with one release fence before arriving and picks up everyone else's with
// one acquire fence after the wait; group leaders pass their group's writes on
// with an acquire-release fence.  The wait polls with relaxed loads, so
// spinning workgroups do not keep invalidating their caches.  gen is the
// number of barriers the grid has passed (every workgroup counts them, and the
// control block starts at zero), so arriving needs no load.  *fend gets the
// next frontier's end.  Returns false if this workgroup's wait timed out (it
// sets ctrl->abort for the summary; any other workgroup still waiting then
// times out too, since the barrier can no longer complete).
__device__ __forceinline__ uint32_t ld_agent(const unsigned int* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(unsigned int* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t add_agent(unsigned int* p, uint32_t v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ bool grid_barrier(Ctrl* ctrl, PeelSync* sy, uint32_t nblocks, uint32_t gen,
                             uint32_t* fend) {
    __shared__ uint32_t s_ok, s_fend;
    // generation (low word) and frontier end (high word), stored and polled
    // as one 64-bit word: a workgroup learns the next frontier's end from the
    // same load that ends its wait
    unsigned long long* const genw = reinterpret_cast<unsigned long long*>(&sy->gen.v[0]);
    // Everything the peel hands from one round to the next goes through
    // agent-scope atomics and coherent loads and stores, so the barrier only
    // has to order: every wave's memory operations complete (s_waitcnt 0)
    // before its workgroup arrives.  Agent-scope fences here wrote back and
    // invalidated the L2 of every workgroup's XCD at every round.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_waitcnt(0);
    lds_barrier();
    if (threadIdx.x == 0) {
        uint32_t ok = 1;
        bool wait = true;
        uint32_t fe = 0;
        // One arrival counter, which only grows (the decode zeroes it once):
        // in barrier gen the last workgroup finds (gen + 1) * nblocks - 1
        // arrivals before its own, reads the queue length and publishes the
        // next generation.  With the fences at workgroup scope one counter
        // beat arrivals in 8 groups plus a top counter (decode NCF 1.422 ->
        // 1.395 ms, VGG19 1.685 -> 1.667 ms, LSTM 1.185 -> 1.162 ms): the
        // group level cost the last arrival one more atomic round trip.
        if (add_agent(&sy->arrive.v[0], 1u) == (gen + 1u) * nblocks - 1u) {
            fe = ld_agent(&sy->tail.v[0]);
            __hip_atomic_store(genw, ((unsigned long long)fe << 32) | (gen + 1u),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            wait = false;
        }
        if (wait) {
            const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
            for (;;) {
                const unsigned long long gw =
                    __hip_atomic_load(genw, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if ((uint32_t)gw != gen) {
                    fe = (uint32_t)(gw >> 32);
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
                if (__builtin_amdgcn_s_memrealtime() - t0 > kBarrierTimeoutTicks) {
                    st_agent(&ctrl->abort, 1u);
                    ok = 0;
                    break;
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        s_ok = ok;
        s_fend = fe;
    }
    lds_barrier();
    *fend = s_fend;
    return s_ok != 0;
}

template <typename T>
__global__ __launch_bounds__(kPeelBlock) void peel_kernel(PeelArgs<T> a) {
    __shared__ PushBuf<kPeelPushCap> q;
    __shared__ uint32_t s_red[2];
    Ctrl* ctrl = a.ctrl;
    PeelSync* sync = a.sync;
    const uint32_t lane = lane_id();
    const uint32_t waves_per_block = kPeelBlock / 64;
    // wave-sized chunks of work go round-robin over the workgroups, so small
    // frontiers still spread over every CU
    const uint32_t gwave = (threadIdx.x >> 6) * gridDim.x + blockIdx.x;
    const uint32_t nwaves = gridDim.x * waves_per_block;
    const bool skip = ctrl->overflow != 0 || ctrl->bad_plan != 0;
    bool ok = true;
    uint32_t my_recovered = 0, my_last_round = 0;
    if (threadIdx.x == 0) {
        q.count = 0;
        s_red[0] = 0;
        s_red[1] = 0;
    }
    lds_barrier();

    if (!skip) {
        const uint32_t nsup = (uint32_t)ctrl->n_support;
        const uint32_t kp = pack_bits(nsup);
        const bool packed = std::is_same<T, int32_t>::value && a.counted && ctrl->nopack == 0;
        if (!a.split0) {
            // round 0's frontier is every cell with exactly one element;
            // packed, each counter also takes its cell's residual in its high
            // word.  Four cells per lane and pass, loaded together, then staged.
            // 64-bit indexes: a sketch of nearly 2^32 cells must not wrap
            const uint64_t nthreads = (uint64_t)gridDim.x * kPeelBlock;
            const uint64_t gtid = (uint64_t)gwave * 64u + lane;
            for (uint64_t base = 0; base < a.cells; base += kScanCells * nthreads) {
                unsigned long long v[kScanCells];
#pragma unroll
                for (uint32_t m = 0; m < kScanCells; m++) {
                    const uint64_t cidx = base + m * nthreads + gtid;
                    v[m] = cidx < a.cells ? a.cnt[cidx] : 0ull;
                }
#pragma unroll
                for (uint32_t m = 0; m < kScanCells; m++) {
                    const uint64_t cidx = base + m * nthreads + gtid;
                    scan_residual(a, cidx, v[m], packed, kp);
                    lds_push(q, (v[m] >> 32) == 1ull, (uint32_t)cidx, (uint32_t)v[m]);
                }
                flush_pushes(q, false, kScanCells * kPeelBlock, &sync->tail.v[0], a.queue,
                             a.cells, a.mark, 1u);
            }
            flush_pushes(q, true, 0, &sync->tail.v[0], a.queue, a.cells, a.mark, 1u);
        }
        // split: round 0 ran before this kernel and the queue holds round 1's
        // frontier after round 0's
        uint32_t fend = 0, gen = 0;
        ok = grid_barrier(ctrl, sync, gridDim.x, gen++, &fend);

        uint32_t qs = a.split0 ? sync->round0.v[0] : 0u;
        if (qs > a.cells) qs = a.cells;
        for (uint32_t r = a.split0 ? 1u : 0u; ok; r++) {
            uint32_t qe = fend;
            if (qe > a.cells) qe = a.cells;  // the queue holds each cell at most once
            if (qe <= qs) break;
            const uint64_t span = (uint64_t)nwaves * 64u;
            const uint32_t nsweep = (uint32_t)(((uint64_t)(qe - qs) + span - 1u) / span);
            for (uint32_t sw = 0; sw < nsweep; sw++) {
                const uint64_t i = qs + ((uint64_t)sw * nwaves + gwave) * 64u + lane;
                bool push[2] = {false, false};
                uint32_t pcell[2] = {0u, 0u}, ppos[2] = {0u, 0u};
                if (i < qe) {
                    // the cell was pure with element pos when queued.  The first
                    // frontier entry of the element to take its flag recovers it;
                    // the flag is already set if it was recovered through another
                    // cell, in this round or an earlier one.  The element and the
                    // cell's residual are read alongside the claim: once claimed,
                    // nothing else changes that cell this round.
                    const unsigned long long qw =
                        ld_agent64(reinterpret_cast<const unsigned long long*>(a.queue + i));
                    const uint2 it = make_uint2((uint32_t)qw, (uint32_t)(qw >> 32));
                    if (it.y < nsup) {
                        bool done = false;
                        if constexpr (std::is_same<T, int32_t>::value) {
                            if (packed) {
                                peel_entry<T, true>(a, it.x, it.y, kp, r, my_recovered,
                                                    my_last_round, push, pcell, ppos);
                                done = true;
                            }
                        }
                        if (!done)
                            peel_entry<T, false>(a, it.x, it.y, kp, r, my_recovered,
                                                 my_last_round, push, pcell, ppos);
                    }
                }
                lds_push(q, push[0], pcell[0], ppos[0]);
                lds_push(q, push[1], pcell[1], ppos[1]);
                flush_pushes(q, false, 2u * kPeelBlock, &sync->tail.v[0], a.queue, a.cells,
                             a.mark, r + 2u);
            }
            flush_pushes(q, true, 0, &sync->tail.v[0], a.queue, a.cells, a.mark, r + 2u);
            qs = qe;
            ok = grid_barrier(ctrl, sync, gridDim.x, gen++, &fend);
        }

    }

    // per-workgroup totals, one atomic each; the last workgroup to finish
    // writes the summary
    my_recovered = wave_sum(my_recovered);
    uint32_t wmax = my_last_round;
    for (int d = 32; d >= 1; d >>= 1) wmax = max(wmax, (uint32_t)__shfl_xor(wmax, d));
    if (lane == 0) {
        atomicAdd(&s_red[0], my_recovered);
        atomicMax(&s_red[1], wmax);
    }
    lds_barrier();
    if (threadIdx.x == 0) {
        if (s_red[0]) atomicAdd(&ctrl->recovered, (unsigned long long)s_red[0]);
        if (s_red[1]) atomicMax(&ctrl->rounds, s_red[1]);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        const uint32_t done = __hip_atomic_fetch_add(&ctrl->done, 1u, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
        if (done == gridDim.x - 1u) {
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            const bool aborted = __hip_atomic_load(&ctrl->abort, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT) != 0;
            const bool overflow = ctrl->overflow != 0;
            const bool bad_plan = ctrl->bad_plan != 0;
            const unsigned long long ns = ctrl->n_support;
            const unsigned long long rec = skip ? 0ull :
                __hip_atomic_load(&ctrl->recovered, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            a.info->n_support = ns;
            a.info->n_recovered = rec;
            a.info->rounds = skip ? 0ull :
                __hip_atomic_load(&ctrl->rounds, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            a.info->success = (!skip && !aborted && rec == ns) ? 1u : 0u;
            a.info->status = bad_plan ? 3u : (overflow ? 1u : (aborted ? 2u : 0u));
        }
    }
}

// ---- round 0 ---------------------------------------------------------------------
//
// For large sketches round 0 runs as ordinary launches over the whole chip,
// the kernel boundaries serving as its barriers: its frontier is large (2.2 M
// entries for VGG19), and the whole chip took it 15-20 % faster than the
// persistent kernel's half grid, which the later, smaller rounds run faster on.
//   scan0    every cell with exactly one element joins round 0's frontier;
//            packed, each counter also takes its cell's residual in its high
//            word.  Four cells per lane and pass, loaded together, then staged;
//   snap0    records where round 0's frontier ends;
//   round0   peels round 0's frontier, appending round 1's to the queue.
constexpr uint32_t kRound0Push = 2048;  // staged entries per workgroup of 256 lanes
// Below this many cells round 0 stays in the persistent kernel: NCF (1.9 M
// cells) and LSTM (6.2 M) lost 16-49 us to the three extra launches, VGG19
// (10.4 M) and BERT-base (11 M) gained about 60 us.
constexpr uint64_t kRound0SplitCells = 8ull << 20;

template <typename T>
__global__ __launch_bounds__(kBlock) void scan0_kernel(PeelArgs<T> a) {
    __shared__ PushBuf<kRound0Push> q;
    const Ctrl* ctrl = a.ctrl;
    if (ctrl->overflow != 0 || ctrl->bad_plan != 0) return;
    if (threadIdx.x == 0) q.count = 0;
    lds_barrier();
    const uint32_t kp = pack_bits((uint32_t)ctrl->n_support);
    const bool packed = std::is_same<T, int32_t>::value && a.counted && ctrl->nopack == 0;
    const uint64_t nthreads = (uint64_t)gridDim.x * kBlock;
    const uint64_t gtid = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    for (uint64_t base = 0; base < a.cells; base += kScanCells * nthreads) {
        unsigned long long v[kScanCells];
#pragma unroll
        for (uint32_t m = 0; m < kScanCells; m++) {
            const uint64_t cidx = base + m * nthreads + gtid;
            v[m] = cidx < a.cells ? a.cnt[cidx] : 0ull;
        }
#pragma unroll
        for (uint32_t m = 0; m < kScanCells; m++) {
            const uint64_t cidx = base + m * nthreads + gtid;
            scan_residual(a, cidx, v[m], packed, kp);
            lds_push(q, (v[m] >> 32) == 1ull, (uint32_t)cidx, (uint32_t)v[m]);
        }
        flush_pushes(q, false, kScanCells * kBlock, &a.sync->tail.v[0], a.queue, a.cells,
                     a.mark, 1u);
    }
    flush_pushes(q, true, 0, &a.sync->tail.v[0], a.queue, a.cells, a.mark, 1u);
}

__global__ void snap0_kernel(PeelSync* sync) {
    if (threadIdx.x == 0) sync->round0.v[0] = sync->tail.v[0];
}

template <typename T>
__global__ __launch_bounds__(kBlock) void round0_kernel(PeelArgs<T> a) {
    __shared__ PushBuf<kRound0Push> q;
    __shared__ uint32_t s_red[2];
    Ctrl* ctrl = a.ctrl;
    if (ctrl->overflow != 0 || ctrl->bad_plan != 0) return;
    if (threadIdx.x == 0) {
        q.count = 0;
        s_red[0] = 0;
        s_red[1] = 0;
    }
    lds_barrier();
    const uint32_t nsup = (uint32_t)ctrl->n_support;
    const uint32_t kp = pack_bits(nsup);
    const bool packed = std::is_same<T, int32_t>::value && a.counted && ctrl->nopack == 0;
    uint32_t qe = a.sync->round0.v[0];
    if (qe > a.cells) qe = a.cells;
    uint32_t my_recovered = 0, my_last_round = 0;
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    for (uint64_t base = 0; base < qe; base += stride) {
        const uint64_t i = base + (uint64_t)blockIdx.x * kBlock + threadIdx.x;
        bool push[2] = {false, false};
        uint32_t pcell[2] = {0u, 0u}, ppos[2] = {0u, 0u};
        if (i < qe) {
            const uint2 it = a.queue[i];
            if (it.y < nsup) {
                bool done = false;
                if constexpr (std::is_same<T, int32_t>::value) {
                    if (packed) {
                        peel_entry<T, true>(a, it.x, it.y, kp, 0u, my_recovered,
                                            my_last_round, push, pcell, ppos);
                        done = true;
                    }
                }
                if (!done)
                    peel_entry<T, false>(a, it.x, it.y, kp, 0u, my_recovered, my_last_round,
                                         push, pcell, ppos);
            }
        }
        lds_push(q, push[0], pcell[0], ppos[0]);
        lds_push(q, push[1], pcell[1], ppos[1]);
        flush_pushes(q, false, 2u * kBlock, &a.sync->tail.v[0], a.queue, a.cells, a.mark, 2u);
    }
    flush_pushes(q, true, 0, &a.sync->tail.v[0], a.queue, a.cells, a.mark, 2u);
    // per-workgroup totals into the control block, summed with the peel's
    my_recovered = wave_sum(my_recovered);
    uint32_t wmax = my_last_round;
    for (int d = 32; d >= 1; d >>= 1) wmax = max(wmax, (uint32_t)__shfl_xor(wmax, d));
    if (lane_id() == 0) {
        atomicAdd(&s_red[0], my_recovered);
        atomicMax(&s_red[1], wmax);
    }
    lds_barrier();
    if (threadIdx.x == 0) {
        if (s_red[0]) atomicAdd(&ctrl->recovered, (unsigned long long)s_red[0]);
        if (s_red[1]) atomicMax(&ctrl->rounds, s_red[1]);
    }
}

// ---- leftovers ---------------------------------------------------------------------

// Algorithm 1's last recovery step for the elements the peel left: the Count
// Sketch median estimate of each one's three cells in the residual sketch
// (from the counters' high words when the peel packed the int32 residuals
// there).  A kernel of its own over the whole chip, not the peel's workgroups:
// when decoding fails most of the support is left, at three scattered loads
// per element.
template <typename T>
__global__ __launch_bounds__(kBlock) void leftover_kernel(PeelArgs<T> a) {
    const Ctrl* ctrl = a.ctrl;
    if (ctrl->overflow != 0 || ctrl->bad_plan != 0) return;
    const uint32_t nsup = (uint32_t)ctrl->n_support;
    // the same test as the peel kernel's
    const bool packed = std::is_same<T, int32_t>::value && a.counted && ctrl->nopack == 0;
    const uint32_t stride = gridDim.x * kBlock;
    for (uint32_t pos = blockIdx.x * kBlock + threadIdx.x; pos < nsup; pos += stride) {
        if (a.peeled[pos]) continue;
        const uint32_t p = a.elem[pos];
        const BatchHash h = batch_hash(a.seed, a.rows, a.cmask, p >> a.log2c);
        const uint32_t t = p & a.cmask;
        T e3[3];
#pragma unroll
        for (int j = 0; j < 3; j++) {
            const uint32_t cell = cell_of(h, j, t, a.c, a.cmask);
            const T y = packed ? (T)(int32_t)(uint32_t)(a.cnt[cell] >> 32) : a.yw[cell];
            e3[j] = Val<T>::sign(y, (h.neg >> j) & 1u);
        }
        a.vals[pos] = median3(e3[0], e3[1], e3[2]);
    }
}

// ---- emit ------------------------------------------------------------------------

template <typename T>
struct EmitArgs {  // T: the gradient type; values are kept in Acc<T>
    const uint32_t* b;
    const uint32_t* blk;
    const uint32_t* elem;
    const typename Acc<T>::type* vals;
    const uint8_t* peeled;
    const T* y_agg;
    const Ctrl* ctrl;
    T* x_out;
    uint32_t* coo_idx;
    T* coo_val;
    uint64_t coo_cap;
    uint32_t* mask;
    uint64_t n, words, seed;
    uint32_t rows, c, cmask, log2c, last_mask;
    bool x_vec;     // x_out is 16-byte aligned
    bool mask_vec;  // mask is 16-byte aligned
    bool b_vec;     // b is 16-byte aligned
};

template <typename T>
__device__ __forceinline__ T estimate_raw(const EmitArgs<T>& a, uint32_t p) {
    const BatchHash h = batch_hash(a.seed, a.rows, a.cmask, p >> a.log2c);
    const uint32_t t = p & a.cmask;
    T e3[3];
#pragma unroll
    for (int j = 0; j < 3; j++)
        e3[j] = Val<T>::sign(a.y_agg[cell_of(h, j, t, a.c, a.cmask)], (h.neg >> j) & 1u);
    return median3(e3[0], e3[1], e3[2]);  // exact in T: a median selects, it does not round
}

// One workgroup per chunk of 1024 bitmap words (32768 parameters).  The
// chunk's members are one contiguous run of E, so their values and recovered
// flags are copied into LDS with coalesced loads, a window of 1024 at a time
// (chunks denser than 1/32 take several): the output loop then has no global
// loads ahead of its stores.  The window sets the workgroup's LDS and so how
// many workgroups a CU keeps writing: measured on MI355X, 1024 members (17 KB,
// eight workgroups per CU) against 2048 (22 KB, seven) took NCF's decode from
// 1.422 to 1.413 ms with VGG19's and LSTM's unchanged, and 4096 cost NCF
// 44 us.  The dense output goes out with nontemporal stores (measured 1-2 %
// faster here, though plain stores win for a pure write stream).
constexpr uint32_t kEmitStage = 1024;  // members per LDS window (1/32 of a chunk's parameters)

template <typename T>
__global__ __launch_bounds__(kBlock) void emit_kernel(EmitArgs<T> a) {
    typedef T V4 __attribute__((ext_vector_type(4)));
    __shared__ uint32_t s_words[kChunkWords];
    __shared__ uint32_t s_pref[kChunkWords];
    __shared__ uint32_t s_mask[kChunkWords];  // the chunk's mask words, stored at the end
    __shared__ uint32_t s_tmp[kBlock / 64];
    __shared__ T s_val[kEmitStage];
    __shared__ uint8_t s_rec[kEmitStage];
    const uint32_t lane = lane_id();
    const uint32_t wave = threadIdx.x >> 6;
    const uint64_t chunk = blockIdx.x;
    const uint64_t w0 = chunk * kChunkWords + 4ull * threadIdx.x;
    const uint4 wv = load_words4(a.b, w0, a.words, a.last_mask, a.b_vec);
    const uint32_t w4[4] = {wv.x, wv.y, wv.z, wv.w};
    const uint32_t mine = __popc(wv.x) + __popc(wv.y) + __popc(wv.z) + __popc(wv.w);
    uint32_t total;
    uint32_t run = block_exclusive_scan(mine, s_tmp, &total);
#pragma unroll
    for (int k = 0; k < 4; k++) {
        s_words[4 * threadIdx.x + k] = w4[k];
        s_pref[4 * threadIdx.x + k] = run;
        run += __popc(w4[k]);
    }
    lds_barrier();
    const uint64_t off = a.blk[chunk];
    // with no valid element list (support over capacity, or a plan for
    // another geometry) every member gets the estimate from the aggregate
    const bool raw = a.ctrl->overflow != 0 || a.ctrl->bad_plan != 0;
    const uint64_t chunk_p = chunk * kChunkBits;
    // the members' values and flags go through LDS in windows of kEmitStage
    // consecutive ranks, [wlo, whi) of the chunk's; an iteration (1024
    // parameters) holds at most 1024 members, so a window that starts at its
    // first member covers it.  wlo, whi and the reload test are uniform.
    uint32_t wlo = 0, whi = 0;
    constexpr uint32_t kIterWords = 4 * kBlock / 32;  // bitmap words per iteration
    for (uint32_t it = 0; it < kChunkBits / (4 * kBlock); it++) {
        if (!raw) {
            const uint32_t wf = it * kIterWords, wl = wf + kIterWords - 1;
            const uint32_t r1 = s_pref[wl] + __popc(s_words[wl]);  // past the iteration's last
            if (r1 > whi) {
                wlo = s_pref[wf];
                whi = wlo + kEmitStage < total ? wlo + kEmitStage : total;
                // the window's loads all in flight together, at indexes
                // clamped to its last member (a reload happens only for an
                // iteration with members, so the window is never empty)
                constexpr uint32_t kPer = kEmitStage / kBlock;
                typename Acc<T>::type v[kPer];
                uint32_t f[kPer];  // not bytes: packing bytes waited for each load
                const uint32_t last = whi > wlo ? whi - 1u : wlo;
#pragma unroll
                for (uint32_t q = 0; q < kPer; q++) {
                    const uint32_t i = wlo + threadIdx.x + q * kBlock;
                    const uint64_t src = off + (i < whi ? i : last);
                    v[q] = a.vals[src];
                    f[q] = a.peeled[src];
                }
                lds_barrier();  // every lane is done with the previous window
#pragma unroll
                for (uint32_t q = 0; q < kPer; q++) {
                    const uint32_t i = wlo + threadIdx.x + q * kBlock;
                    if (i < whi) {
                        s_val[i - wlo] = (T)v[q];
                        s_rec[i - wlo] = f[q] != 0u ? 1 : 0;
                    }
                }
                lds_barrier();
            }
        }
        const uint32_t e0 = it * (4 * kBlock) + 4u * threadIdx.x;  // offset in the chunk
        const uint64_t p0 = chunk_p + e0;
        const uint32_t wi = e0 >> 5, sh = e0 & 31u;
        const uint32_t word = s_words[wi];
        uint64_t rank = off + s_pref[wi] + __popc(word & ((1u << sh) - 1u));
        T out[4];
        bool rec[4];
#pragma unroll
        for (int k = 0; k < 4; k++) {
            out[k] = T(0);
            rec[k] = false;
            if ((word >> (sh + k)) & 1u) {
                const uint32_t p = (uint32_t)(p0 + k);
                if (!raw) {
                    out[k] = s_val[rank - off - wlo];
                    rec[k] = s_rec[rank - off - wlo] != 0;
                } else {
                    out[k] = estimate_raw(a, p);
                }
                if (a.coo_idx != nullptr && rank < a.coo_cap) {
                    a.coo_idx[rank] = p;
                    a.coo_val[rank] = out[k];
                }
                rank++;
            }
        }
        if (a.x_out != nullptr && p0 < a.n) {
            if (a.x_vec && p0 + 4 <= a.n) {
                V4 v = {out[0], out[1], out[2], out[3]};
                __builtin_nontemporal_store(v, reinterpret_cast<V4*>(a.x_out + p0));
            } else {
                for (int k = 0; k < 4; k++)
                    if (p0 + k < a.n) a.x_out[p0 + k] = out[k];
            }
        }
        if (a.mask != nullptr) {
            const uint64_t m0 = __ballot(rec[0]), m1 = __ballot(rec[1]);
            const uint64_t m2 = __ballot(rec[2]), m3 = __ballot(rec[3]);
            if (lane < 8) {
                const uint32_t s8 = 8u * lane;
                const uint32_t mw = spread4((uint32_t)(m0 >> s8)) |
                                    (spread4((uint32_t)(m1 >> s8)) << 1) |
                                    (spread4((uint32_t)(m2 >> s8)) << 2) |
                                    (spread4((uint32_t)(m3 >> s8)) << 3);
                s_mask[((it * (4 * kBlock) + wave * 256u) >> 5) + lane] = mw;
            }
        }
    }
    if (a.mask != nullptr) {
        // one 16-byte store per lane instead of a 4-byte store by 8 lanes per
        // wave and iteration
        lds_barrier();
        const uint64_t mw0 = chunk * kChunkWords + 4ull * threadIdx.x;
        if (a.mask_vec && mw0 + 4 <= a.words) {
            *reinterpret_cast<uint4*>(a.mask + mw0) =
                make_uint4(s_mask[4 * threadIdx.x], s_mask[4 * threadIdx.x + 1],
                           s_mask[4 * threadIdx.x + 2], s_mask[4 * threadIdx.x + 3]);
        } else {
            for (uint32_t k = 0; k < 4; k++)
                if (mw0 + k < a.words) a.mask[mw0 + k] = s_mask[4 * threadIdx.x + k];
        }
    }
}

// Section 3.3 query: parameter p is a candidate iff its k filter bits are all
// set.  One lane per candidate word (32 parameters).  For c >= 32 the word lies
// in one batch, and under hash i its 32 bits sit rotated in one filter row:
// the two filter words covering them, shifted back by the rotation, give the
// hash's 32 answers at once; the word is their AND over i (stopping once it is
// zero).  Below c = 32 each parameter is checked bit by bit.
__global__ __launch_bounds__(kBlock) void bloom_probe_kernel(
    const uint32_t* __restrict__ f, uint32_t* __restrict__ cand, uint64_t n, uint64_t words,
    uint64_t seed, uint32_t k, uint32_t brows, uint32_t c, uint32_t cmask, uint32_t log2c,
    uint32_t last_mask) {
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    for (uint64_t w = (uint64_t)blockIdx.x * kBlock + threadIdx.x; w < words; w += stride) {
        const uint64_t p0 = w << 5;
        uint32_t acc;
        if (c >= 32) {
            const uint64_t b = p0 >> log2c;
            const uint32_t cw = c >> 5, ow = ((uint32_t)p0 & cmask) >> 5;
            acc = ~0u;
            for (uint32_t i = 0; i < k && acc != 0u; i++) {
                const BloomHash h = bloom_hash(seed, k, brows, cmask, b, i);
                const uint32_t q = h.bias >> 5, r = h.bias & 31u;
                const uint32_t* rp = f + (uint64_t)h.row * cw;
                const uint32_t w0 = (ow + q) & (cw - 1u);
                uint32_t v = rp[w0] >> r;
                if (r != 0u) v |= rp[(w0 + 1u) & (cw - 1u)] << (32u - r);
                acc &= v;
            }
        } else {
            acc = 0u;
            for (uint32_t sb = 0; sb < 32; sb++) {
                const uint64_t p = p0 + sb;
                if (p >= n) break;
                const uint64_t b = p >> log2c;
                const uint32_t t = (uint32_t)p & cmask;
                bool all = true;
                for (uint32_t i = 0; i < k && all; i++) {
                    const BloomHash h = bloom_hash(seed, k, brows, cmask, b, i);
                    const uint32_t bit = h.row * c + ((t + h.bias) & cmask);
                    all = ((f[bit >> 5] >> (bit & 31u)) & 1u) != 0u;
                }
                acc |= (all ? 1u : 0u) << sb;
            }
        }
        if (w == words - 1) acc &= last_mask;
        cand[w] = acc;
    }
}

template <typename T>
hipError_t launch_decode_t(const Geo& g, const void* plan, const void* y_agg_v,
                           const uint32_t* b, const DecodeOut& out, const DecodeLayout& L,
                           void* ws, hipStream_t s) {
    char* base = static_cast<char*>(ws);
    typedef typename Acc<T>::type A;
    Ctrl* ctrl = reinterpret_cast<Ctrl*>(base + L.ctrl);
    PeelSync* sync = reinterpret_cast<PeelSync*>(base + L.sync);
    uint32_t* blk = reinterpret_cast<uint32_t*>(base + L.blk);
    uint32_t* tcnt = reinterpret_cast<uint32_t*>(base + L.tcnt);
    uint32_t* cpre = reinterpret_cast<uint32_t*>(base + L.cpre);
    uint32_t* woffb = plan ? reinterpret_cast<uint32_t*>(base + L.woffb) : nullptr;
    uint32_t* elem = reinterpret_cast<uint32_t*>(base + L.elem);
    A* vals = reinterpret_cast<A*>(base + L.vals);
    uint8_t* peeled = reinterpret_cast<uint8_t*>(base + L.peeled);
    unsigned long long* cnt = reinterpret_cast<unsigned long long*>(base + L.cnt);
    A* yw = reinterpret_cast<A*>(base + L.yw);
    uint2* queue = reinterpret_cast<uint2*>(base + L.queue);
    uint32_t* mark = g.f32 ? reinterpret_cast<uint32_t*>(base + L.mark) : nullptr;
    const T* y_agg = static_cast<const T*>(y_agg_v);
    const bool planned = plan != nullptr;

    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;

    uint64_t grid = ((uint64_t)g.cells + kBlock - 1) / kBlock;
    if (grid > (uint64_t)di.cus * 16) grid = (uint64_t)di.cus * 16;
    hipLaunchKernelGGL(prep_kernel<T>, dim3((uint32_t)grid), dim3(kBlock), 0, s, y_agg, yw, cnt,
                       g.cells, planned, ctrl, sync, mark);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const uint32_t last_mask = (g.n & 31u) ? ((1u << (g.n & 31u)) - 1u) : 0xffffffffu;
    const bool bvec = (reinterpret_cast<uintptr_t>(b) & 15u) == 0;
    hipLaunchKernelGGL(tile_count_kernel, dim3((uint32_t)L.ntiles), dim3(kBlock), 0, s, b,
                       g.words, last_mask, bvec, L.nchunks, cpre, tcnt);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(1024), 0, s, tcnt, L.ntiles, ctrl, L.cap);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    SupportArgs sa;
    sa.b = b;
    sa.cpre = cpre;
    sa.toff = tcnt;
    sa.blk = blk;
    sa.woffb = woffb;
    sa.elem = elem;
    sa.peeled = peeled;
    sa.cnt = cnt;
    sa.ctrl = ctrl;
    sa.words = g.words;
    sa.nchunks = L.nchunks;
    sa.cap = L.cap;
    sa.seed = g.seed;
    sa.last_mask = last_mask;
    sa.log2wpb = planned ? g.log2c - 5u : 0u;  // planned sketches have c >= 256
    sa.nb = (uint32_t)((g.n + g.c - 1) / g.c);
    sa.rows = g.rows;
    sa.c = g.c;
    sa.cmask = g.cmask;
    sa.log2c = g.log2c;
    sa.vec = bvec;
    hipLaunchKernelGGL(support_kernel, dim3((uint32_t)((L.nchunks + kBlock / 64 - 1) / (kBlock / 64))),
                       dim3(kBlock), 0, s, sa);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    // A wave per row when rows are to spare (two or more per SIMD); then, for
    // int32, round 0 as two passes over the rows (pure_rows, round0_rows)
    // instead of the counter kernel and the entry-by-entry round, and the peel
    // kernel starts from round 1 (LSTM, 6.2 M cells: decode 1.40 -> 1.32 ms).
    const bool wave_rows = planned && (uint64_t)g.rows >= 8ull * (uint64_t)di.cus;
    // Round 0 by rows works through every member of every live batch twice;
    // it pays when the sketch has at least a cell per support element (the
    // decode's support bound), where it replaces the entry-by-entry round 0.
    // Below that the sketch cannot peel anyway and round 0 recovers little:
    // on section 4.1's VGG19 gradient (69.6 % dense) at sketch sizes of 0.02
    // to 0.6 of n the decode took 2.35-3.68 ms by rows against 1.18-3.37 ms
    // without, and from 0.7 up 4.78-7.57 ms against 4.85-14.5 ms.
    const bool rows0 = wave_rows && std::is_same<T, int32_t>::value && (uint64_t)g.cells >= L.cap;
    Round0Args ra;
    ra.y_agg = reinterpret_cast<const int32_t*>(y_agg_v);
    ra.vals = reinterpret_cast<int32_t*>(vals);
    ra.peeled = peeled;
    ra.elem = elem;
    ra.yw = reinterpret_cast<int32_t*>(yw);
    ra.queue = queue;
    ra.tail = &sync->tail.v[0];
    ra.log2c = g.log2c;
    // one wave per row over the whole chip, as many workgroups as fit
    auto launch_rows = [&](auto k1024, auto k512, auto k256, auto args) -> hipError_t {
        const void* kfn = g.c == 1024 ? reinterpret_cast<const void*>(k1024)
                        : g.c == 512 ? reinterpret_cast<const void*>(k512)
                                     : reinterpret_cast<const void*>(k256);
        int per_cu = 0;
        hipError_t err = occupancy_per_cu(kfn, kBlock, &per_cu);
        if (err != hipSuccess) return err;
        const uint64_t want = ((uint64_t)g.rows + kBlock / 64 - 1) / (kBlock / 64);
        const uint64_t cap = (uint64_t)di.cus * per_cu;
        const uint32_t cgrid = (uint32_t)(want < cap ? want : cap);
        if (g.c == 1024)
            hipLaunchKernelGGL(k1024, dim3(cgrid), dim3(kBlock), 0, s, args);
        else if (g.c == 512)
            hipLaunchKernelGGL(k512, dim3(cgrid), dim3(kBlock), 0, s, args);
        else
            hipLaunchKernelGGL(k256, dim3(cgrid), dim3(kBlock), 0, s, args);
        return hipGetLastError();
    };

    if (planned) {
        const PlanLayout PL = plan_layout(g);
        const char* pb = static_cast<const char*>(plan);
        CounterArgs ca;
        ca.hdr = reinterpret_cast<const PlanHeader*>(pb + PL.header);
        ca.rowoff = reinterpret_cast<const uint32_t*>(pb + PL.rowoff);
        ca.entry = reinterpret_cast<const uint2*>(pb + PL.entry);
        ca.b = b;
        ca.woffb = woffb;
        ca.cnt = cnt;
        ca.ctrl = ctrl;
        ca.n = g.n;
        ca.seed = g.seed;
        ca.words = g.words;
        ca.nb = PL.nb;
        ca.rows = g.rows;
        ca.c = g.c;
        ca.cmask = g.cmask;
        ca.cells = g.cells;
        ca.last_mask = last_mask;
        // Rows to spare (two or more per SIMD): one wave per row, its loads in
        // flight together.  Fewer, longer rows (NCF: 1.9 K rows of 1.7 K plan
        // entries) keep more waves busy as a workgroup per row, or, when a
        // row has only a few entries, a wave per row walking them in turn.
        if (rows0) {
            ra.c = ca;
            if ((e = launch_rows(pure_rows_kernel<1024>, pure_rows_kernel<512>,
                                 pure_rows_kernel<256>, ra)) != hipSuccess)
                return e;
        } else if (wave_rows) {
            if ((e = launch_rows(counter_rows_kernel<1024>, counter_rows_kernel<512>,
                                 counter_rows_kernel<256>, ca)) != hipSuccess)
                return e;
        } else if (3ull * ((g.n + g.c - 1) / g.c) <= kWaveRowsEntries * g.rows) {
            const uint64_t want = ((uint64_t)g.rows + 3) / 4;  // four waves per workgroup
            const uint32_t cgrid = want < (uint64_t)di.cus * 8 ? (uint32_t)want : (uint32_t)di.cus * 8;
            if (g.c == 1024)
                hipLaunchKernelGGL(counter_wave_kernel<1024>, dim3(cgrid), dim3(kBlock), 0, s, ca);
            else if (g.c == 512)
                hipLaunchKernelGGL(counter_wave_kernel<512>, dim3(cgrid), dim3(kBlock), 0, s, ca);
            else
                hipLaunchKernelGGL(counter_wave_kernel<256>, dim3(cgrid), dim3(kBlock), 0, s, ca);
        } else {
            const uint32_t cgrid = g.rows < (uint32_t)di.cus * 8 ? g.rows : (uint32_t)di.cus * 8;
            if (g.c == 1024)
                hipLaunchKernelGGL(counter_kernel<1024>, dim3(cgrid), dim3(kBlock), 0, s, ca);
            else if (g.c == 512)
                hipLaunchKernelGGL(counter_kernel<512>, dim3(cgrid), dim3(kBlock), 0, s, ca);
            else
                hipLaunchKernelGGL(counter_kernel<256>, dim3(cgrid), dim3(kBlock), 0, s, ca);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }

    // persistent peel: every workgroup must be resident (cooperative launch);
    // one per CU at most, so it is enough that one fits
    int per_cu = 0;
    e = occupancy_per_cu(reinterpret_cast<const void*>(&peel_kernel<A>), kPeelBlock, &per_cu);
    if (e != hipSuccess) return e;
    // At most one resident workgroup per CU.  A round costs a fixed barrier
    // time that grows with the number of workgroups arriving (about 6.9 us at
    // one per CU, 4.9 us at one per two CUs on MI355X) plus a per-entry time
    // bound by the atomics the CUs can keep in flight (about 10 % higher on
    // half the CUs).  Rounds are about 50-65 at the default sketch ratio, so
    // a small sketch, with few entries per round, peels faster on half the
    // CUs and a large one on all of them; with five atomics per element the
    // two meet near 8 M cells.  The int32 peel with a plan (residuals in the
    // counters, three atomics per element) measured faster on half the CUs up
    // to 11 M cells, and slower at 97 M (BERT-base at 5 %: 16.1 against
    // 18.3 ms).
    // With the barrier's fences at workgroup scope (a cheaper round), the
    // int32 peel with a plan measured fastest on three quarters of the CUs
    // from 8 M cells up to that bound (VGG19, 10.4 M cells: 1.727 -> 1.683 ms;
    // BERT-base, 11.0 M: 1.794 -> 1.742 ms) and still on half below it (NCF
    // 1.417 against 1.425 ms; LSTM 1.167 against 1.177 ms).
    const bool fewer_atomics = std::is_same<T, int32_t>::value && planned;
    const uint64_t half_below = fewer_atomics ? kPeelHalfGridCellsInt : kPeelHalfGridCells;
    uint32_t peel_grid = g.cells < half_below && di.cus >= 2 ? (uint32_t)di.cus / 2u
                                                             : (uint32_t)di.cus;
    if (fewer_atomics && g.cells >= kPeelHalfGridCells && g.cells < half_below && di.cus >= 4)
        peel_grid = (uint32_t)di.cus / 4u * 3u;
    PeelArgs<A> pa;
    pa.ctrl = ctrl;
    pa.sync = sync;
    pa.elem = elem;
    pa.vals = vals;
    pa.peeled = peeled;
    pa.cnt = cnt;
    pa.yw = yw;
    pa.y_agg = g.f32 ? nullptr : static_cast<const int32_t*>(y_agg_v);
    pa.queue = queue;
    pa.mark = mark;
    pa.info = static_cast<InfoDev*>(out.info);
    pa.seed = g.seed;
    pa.rows = g.rows;
    pa.c = g.c;
    pa.cmask = g.cmask;
    pa.log2c = g.log2c;
    pa.cells = g.cells;
    pa.counted = planned;
    // large sketches (large round-0 frontiers) take round 0 on the whole chip
    pa.split0 = rows0 || g.cells >= kRound0SplitCells;  // round 0 ran before the peel kernel
    if (rows0) {
        if ((e = launch_rows(round0_rows_kernel<1024>, round0_rows_kernel<512>,
                             round0_rows_kernel<256>, ra)) != hipSuccess)
            return e;
    } else if (pa.split0) {
        const uint32_t grid0 = (uint32_t)di.cus * 8;
        hipLaunchKernelGGL(scan0_kernel<A>, dim3(grid0), dim3(kBlock), 0, s, pa);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(snap0_kernel, dim3(1), dim3(64), 0, s, sync);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(round0_kernel<A>, dim3(grid0), dim3(kBlock), 0, s, pa);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    void* args[] = {&pa};
    e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(&peel_kernel<A>),
                                   dim3(peel_grid), dim3(kPeelBlock), args,
                                   0, s);
    if (e != hipSuccess) return e;

    if (out.x_out != nullptr || out.mask != nullptr || out.coo_idx != nullptr) {
        hipLaunchKernelGGL(leftover_kernel<A>, dim3((uint32_t)di.cus * 8), dim3(kBlock), 0, s, pa);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        EmitArgs<T> ea;
        ea.b = b;
        ea.blk = blk;
        ea.elem = elem;
        ea.vals = vals;
        ea.peeled = peeled;
        ea.y_agg = y_agg;
        ea.ctrl = ctrl;
        ea.x_out = static_cast<T*>(out.x_out);
        ea.coo_idx = out.coo_idx;
        ea.coo_val = static_cast<T*>(out.coo_val);
        ea.coo_cap = out.coo_idx != nullptr && out.coo_val != nullptr ? out.coo_cap : 0;
        if (ea.coo_cap == 0) ea.coo_idx = nullptr;
        ea.mask = out.mask;
        ea.n = g.n;
        ea.words = g.words;
        ea.seed = g.seed;
        ea.rows = g.rows;
        ea.c = g.c;
        ea.cmask = g.cmask;
        ea.log2c = g.log2c;
        ea.last_mask = last_mask;
        ea.x_vec = (reinterpret_cast<uintptr_t>(out.x_out) & 15u) == 0;
        ea.mask_vec = (reinterpret_cast<uintptr_t>(out.mask) & 15u) == 0;
        ea.b_vec = bvec;
        hipLaunchKernelGGL(emit_kernel<T>, dim3((uint32_t)L.nchunks), dim3(kBlock), 0, s, ea);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

}  // namespace

DecodeLayout decode_layout(const Geo& g, uint64_t max_support) {
    DecodeLayout L;
    uint64_t cap = max_support == 0 ? g.n : max_support;
    if (cap > g.n) cap = g.n;
    if (cap > 0x7fffffffull) cap = 0x7fffffffull;  // packed counters need |S| < 2^31
    L.cap = cap;
    L.nchunks = (g.words + kChunkWords - 1) / kChunkWords;
    const size_t vsz = g.f32 ? 8 : 4;  // decode-side values: int32, or fp64 for fp32
    size_t o = 0;
    L.ctrl = o;    o = align256(o + sizeof(Ctrl));
    L.sync = o;    o = align256(o + sizeof(PeelSync));
    L.ntiles = (L.nchunks + kTileChunks - 1) / kTileChunks;
    L.blk = o;     o = align256(o + L.nchunks * 4);
    L.cpre = o;    o = align256(o + L.nchunks * 4);
    L.tcnt = o;    o = align256(o + L.ntiles * 4);
    // rank offsets per batch of c parameters, used with a plan (c >= 256)
    L.woffb = o;   o = align256(o + (g.c >= 256 ? ((g.n + g.c - 1) / g.c + 1) * 4 : 0));
    L.elem = o;    o = align256(o + cap * 4);
    L.vals = o;    o = align256(o + cap * vsz);
    L.peeled = o;  o = align256(o + cap);  // a byte per element
    L.cnt = o;     o = align256(o + (size_t)g.cells * 8);
    L.yw = o;      o = align256(o + (size_t)g.cells * vsz);
    L.queue = o;   o = align256(o + (size_t)g.cells * 8);
    L.mark = o;    o = align256(o + (g.f32 ? (size_t)g.cells * 4 : 0));  // fp32: frontier marks
    L.cand = o;    o = align256(o + (g.bloom_k ? g.words * 4 : 0));  // probed Bloom candidates
    L.total = o;
    return L;
}

hipError_t launch_bloom_probe(const Geo& g, const uint32_t* filter, uint32_t* cand,
                              hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    uint64_t grid = (g.words + kBlock - 1) / kBlock;
    if (grid > (uint64_t)di.cus * 16) grid = (uint64_t)di.cus * 16;
    const uint32_t last_mask = (g.n & 31u) ? ((1u << (g.n & 31u)) - 1u) : 0xffffffffu;
    hipLaunchKernelGGL(bloom_probe_kernel, dim3((uint32_t)grid), dim3(kBlock), 0, s, filter,
                       cand, g.n, g.words, g.seed, g.bloom_k, g.bloom_rows, g.c, g.cmask,
                       g.log2c, last_mask);
    return hipGetLastError();
}

hipError_t launch_support_offsets(const Geo& g, const uint32_t* b, uint32_t* blk, void* ctrl,
                                  hipStream_t s) {
    const uint64_t nchunks = (g.words + kChunkWords - 1) / kChunkWords;
    const uint32_t last_mask = (g.n & 31u) ? ((1u << (g.n & 31u)) - 1u) : 0xffffffffu;
    Ctrl* c = static_cast<Ctrl*>(ctrl);
    hipLaunchKernelGGL(count_kernel, dim3((uint32_t)nchunks), dim3(kBlock), 0, s, b, g.words,
                       last_mask, blk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(1024), 0, s, blk, nchunks, c, g.n);
    return hipGetLastError();
}

hipError_t launch_decode(const Geo& g, const void* plan, const void* y_agg, const uint32_t* b_agg,
                         const DecodeOut& out, const DecodeLayout& L, void* ws, hipStream_t s) {
    if (g.bloom_k != 0) {
        // the support is what the filter reports: probe it into a bitmap of
        // candidates, then decode as with the bitmap index
        uint32_t* cand = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + L.cand);
        const hipError_t e = launch_bloom_probe(g, b_agg, cand, s);
        if (e != hipSuccess) return e;
        b_agg = cand;
    }
    if (g.f32) return launch_decode_t<float>(g, plan, y_agg, b_agg, out, L, ws, s);
    return launch_decode_t<int32_t>(g, plan, y_agg, b_agg, out, L, ws, s);
}

}  // namespace hc
