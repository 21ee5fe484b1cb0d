// hc_encode.hip -- worker-side compression (Algorithm 1, phase I) for gfx950.
//
// Dense path.  Each wave takes tiles of 1024 consecutive parameters, read as
// four coalesced 16-byte nontemporal loads per lane (the gradient is read
// once, so it should not evict the sketch from L2/MALL).  Per tile:
//   - sixteen ballots of "x != 0" become the tile's 32 bitmap words (section
//     3.2); only the nonzero words are stored, into a bitmap zero-filled by a
//     pure write pass before the kernel (on MI355X, bitmap stores interleaved
//     with the 4n-byte read stream cost about 0.18 ms per 2^30 parameters
//     however they are shaped, against 0.02 ms for the separate fill);
//   - every nonzero adds g_j * x to its three cells (section 3.1) with
//     fire-and-forget global atomics.  Within one batch the cells of a hash
//     are one sketch row rotated by a bias (section 3.4), so the atomics of a
//     load land in at most three 4 KiB rows.
// The batch hash is wave-uniform when c >= 256 (computed on the scalar unit
// once per wave and tile), per lane when 4 <= c < 256, per element below.
#include <type_traits>

#include "hc_device.h"
#include "hc_internal.h"

namespace hc {

namespace {

constexpr int kBlock = 256;
constexpr uint64_t kTile = 1024;  // parameters per wave tile

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

template <typename T> struct Vec4;
template <> struct Vec4<int32_t> { typedef v4i type; };
template <> struct Vec4<float> { typedef v4f type; };

// Sets p[0, count) to value; vec: p is 16-byte aligned (else plain 4-byte
// stores throughout).  Workgroups [0, g0) fill p, the rest fill p2[0, count2)
// (p2 may be null): one launch clears both of an encode's outputs.  Each
// workgroup fills one contiguous run of kFillVecs 16-byte vectors (a 4 GiB
// store stream measured 0.730 ms this way, 0.87-1.04 ms grid-strided).
constexpr uint64_t kFillVecs = 8192;  // 128 KiB per workgroup
__device__ __forceinline__ void fill_range(uint32_t* __restrict__ p, uint64_t count,
                                           uint32_t value, bool vec, uint32_t blk,
                                           uint32_t nblk) {
    if (!vec) {
        const uint64_t stride = (uint64_t)nblk * kBlock;
        for (uint64_t i = (uint64_t)blk * kBlock + threadIdx.x; i < count; i += stride)
            p[i] = value;
        return;
    }
    const uint64_t nvec = count / 4;
    const uint64_t v0 = (uint64_t)blk * kFillVecs;
    const uint64_t v1 = v0 + kFillVecs < nvec ? v0 + kFillVecs : nvec;
    const v4u v = {value, value, value, value};
    for (uint64_t i = v0 + threadIdx.x; i < v1; i += kBlock) reinterpret_cast<v4u*>(p)[i] = v;
    if (blk == 0 && threadIdx.x < count - nvec * 4) p[nvec * 4 + threadIdx.x] = value;
}

__global__ __launch_bounds__(kBlock) void fill_u32_kernel(uint32_t* __restrict__ p,
                                                          uint64_t count, bool vec,
                                                          uint32_t* __restrict__ p2,
                                                          uint64_t count2, bool vec2,
                                                          uint32_t g0, uint32_t value) {
    if (blockIdx.x < g0)
        fill_range(p, count, value, vec, blockIdx.x, g0);
    else
        fill_range(p2, count2, value, vec2, blockIdx.x - g0, gridDim.x - g0);
}

// Sketch updates for the parameters of one load: e[k] is parameter p0 + k of
// this lane, p0 = lbase + 4 * lane, lbase the load's first parameter.  rows:
// the sketch's rows, or a blocked sketch's rows per block (block: its batches
// per block, 0 for the global sketch).
template <typename T, int MODE>
__device__ __forceinline__ void scatter_load(const T (&e)[4], const bool (&nz)[4], uint64_t lbase,
                                             uint64_t p0, T* __restrict__ y, uint64_t seed,
                                             uint32_t rows, uint32_t block, uint32_t c,
                                             uint32_t cmask, uint32_t log2c) {
    if (MODE == 0) {
        const BatchHash h =
            batch_hash_blocked(seed, rows, cmask, log2c, uniform64(lbase >> log2c), block);
        if (nz[0] | nz[1] | nz[2] | nz[3]) {
#pragma unroll
            for (int k = 0; k < 4; k++) {
                if (!nz[k]) continue;
                const uint32_t t = (uint32_t)(p0 + k) & cmask;
#pragma unroll
                for (int j = 0; j < 3; j++)
                    Val<T>::atomic_add(y + cell_of(h, j, t, c, cmask),
                                       Val<T>::sign(e[k], (h.neg >> j) & 1u));
            }
        }
    } else if (MODE == 1) {
        if (nz[0] | nz[1] | nz[2] | nz[3]) {
            const BatchHash h = batch_hash_blocked(seed, rows, cmask, log2c, p0 >> log2c, block);
#pragma unroll
            for (int k = 0; k < 4; k++) {
                if (!nz[k]) continue;
                const uint32_t t = (uint32_t)(p0 + k) & cmask;
#pragma unroll
                for (int j = 0; j < 3; j++)
                    Val<T>::atomic_add(y + cell_of(h, j, t, c, cmask),
                                       Val<T>::sign(e[k], (h.neg >> j) & 1u));
            }
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; k++) {
            if (!nz[k]) continue;
            const uint64_t p = p0 + k;
            const BatchHash h = batch_hash_blocked(seed, rows, cmask, log2c, p >> log2c, block);
            const uint32_t t = (uint32_t)p & cmask;
#pragma unroll
            for (int j = 0; j < 3; j++)
                Val<T>::atomic_add(y + cell_of(h, j, t, c, cmask),
                                   Val<T>::sign(e[k], (h.neg >> j) & 1u));
        }
    }
}

// Staged encode, first pass: the nonzeros of every batch of c >= 256
// parameters go to the batch's list of kStageCap (column, value) entries in
// the staging buffer, at ranks taken from the wave's ballots; count[b] gets
// the batch's number of nonzeros (the lists keep the first kStageCap; a batch
// with more is read from the gradient itself by the second pass).  No global
// atomics: the sketch is assembled row by row afterwards.
struct StageOut {
    uint2* list;      // [nb * kStageCap]: .x = column t, .y = value bits
    uint32_t* count;  // [nb]
    uint64_t nb;      // batches: a tile past the gradient's end names batches >= nb
};

template <typename T>
__device__ __forceinline__ uint32_t value_bits(T v) {
    return __builtin_bit_cast(uint32_t, v);
}

// The wave's staged entries of batch b (cnt nonzeros, the first kStageCap in
// stage[]) go to the batch's list with one store, lane r storing entry r.
// Every batch's count is written, zero or not (the staged encode clears
// nothing beforehand).
static_assert(kStageCap == 64, "one staged entry per lane");
__device__ __forceinline__ void flush_batch(const uint2* stage, uint32_t cnt, uint64_t b,
                                            uint32_t lane, const StageOut& so) {
    if (lane == 0 && b < so.nb) so.count[b] = cnt;
    if (cnt == 0u) return;  // uniform over the wave (a batch >= nb has none)
    __builtin_amdgcn_s_waitcnt(0xc07f);  // the wave's LDS writes have landed
    __builtin_amdgcn_wave_barrier();
    if (lane < cnt) so.list[b * kStageCap + lane] = stage[lane];
    __builtin_amdgcn_s_waitcnt(0xc07f);  // read back before the stage is refilled
    __builtin_amdgcn_wave_barrier();
}

// e[l][k] is parameter tbase + 256 l + 4 lane + k; a batch spans c / 256
// loads.  Each nonzero's (column, value) goes to the wave's LDS stage at its
// rank in the batch, and each batch's run is then stored whole.
template <typename T>
__device__ __forceinline__ void stage_tile(const T (&e)[4][4], const bool (&nz)[4][4],
                                           const uint64_t (&m)[4][4], uint64_t tbase,
                                           uint32_t lane, const StageOut& so, uint32_t log2c,
                                           uint2* stage) {
    const uint32_t cmask = (1u << log2c) - 1u;
    uint32_t base = 0;  // nonzeros of the current batch before this load
#pragma unroll
    for (int l = 0; l < 4; l++) {
        const uint64_t pl = tbase + 256ull * l;
        if (l > 0 && (pl & cmask) == 0u) {  // load l starts a new batch
            flush_batch(stage, base, (pl >> log2c) - 1u, lane, so);
            base = 0;
        }
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const uint64_t mk = m[l][k];
            if (mk == 0ull) continue;  // uniform over the wave
            if (nz[l][k]) {
                const uint32_t rank = base + lanes_below(mk);
                if (rank < kStageCap)
                    stage[rank] = make_uint2((256u * (uint32_t)l + 4u * lane + (uint32_t)k) & cmask,
                                             value_bits(e[l][k]));
            }
            base += (uint32_t)__popcll(mk);
        }
    }
    flush_batch(stage, base, (tbase + 768u) >> log2c, lane, so);
}

// One wave tile: 1024 consecutive parameters from `tbase` (a multiple of
// 1024), four loads of 256 per wave, e[l][k] = parameter tbase + 256 l +
// 4 lane + k.  Its 32 bitmap words are built from the 16 ballots in lanes
// 0..31, which store the nonzero ones (the bitmap was zero-filled); with a
// Bloom-filter index (BL) each nonzero word is OR-ed, rotated, into the filter
// instead (section 3.3).
template <typename T, int MODE, bool BL, bool STAGED>
__device__ __forceinline__ void encode_tile(const T (&e)[4][4], uint64_t tbase, uint32_t lane,
                                            T* __restrict__ y, uint32_t* __restrict__ b,
                                            uint64_t words, uint64_t seed, uint32_t rows,
                                            uint32_t block, uint32_t c, uint32_t cmask,
                                            uint32_t log2c, uint32_t bk, uint32_t brows,
                                            const StageOut& so, uint2* stage) {
    bool nz[4][4];
    uint64_t m[4][4], any = 0;
#pragma unroll
    for (int l = 0; l < 4; l++)
#pragma unroll
        for (int k = 0; k < 4; k++) {
            nz[l][k] = Val<T>::nonzero(e[l][k]);
            m[l][k] = __ballot(nz[l][k]);
            any |= m[l][k];
        }
    // an all-zero tile has nothing to store (the bitmap was zero-filled) and
    // nothing to add: on a sparse gradient that is almost every tile, and
    // skipping the word assembly keeps the wave's next loads coming sooner.
    // The staged encode clears nothing beforehand and stores every tile's
    // words and counts, zero or not.
    if (!STAGED && any == 0) return;
    // word w = 8 l + i holds parameters 32 w .. 32 w + 31: lanes 8i..8i+7 of
    // load l, parameter 4 lane' + k at bit 4 (lane' - 8 i) + k
    if (lane < 32) {
        const uint32_t l = lane >> 3, sh = 8u * (lane & 7u);
        uint32_t word = 0;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const uint64_t mk = l == 0 ? m[0][k] : l == 1 ? m[1][k] : l == 2 ? m[2][k] : m[3][k];
            word |= spread4((uint32_t)(mk >> sh)) << k;
        }
        const uint64_t widx = (tbase >> 5) + lane;
        if (!BL) {
            // staged: all 32 words of every tile, one full 128-byte line
            if ((STAGED || word != 0u) && widx < words) b[widx] = word;
        } else if (word != 0u) {
            bloom_insert_word(b, word, widx << 5, seed, bk, brows, c, cmask, log2c);
        }
    }
    if (STAGED) {
        stage_tile<T>(e, nz, m, tbase, lane, so, log2c, stage);
        return;
    }
#pragma unroll
    for (int l = 0; l < 4; l++) {
        if ((m[l][0] | m[l][1] | m[l][2] | m[l][3]) == 0) continue;
        const uint64_t lbase = tbase + 256ull * l;
        scatter_load<T, MODE>(e[l], nz[l], lbase, lbase + 4ull * lane, y, seed, rows, block, c,
                              cmask, log2c);
    }
}

// MODE 0: c >= 256 (the batch is uniform over a load: hash on the scalar
// unit), MODE 1: 4 <= c < 256 (per lane), MODE 2: c < 4 (per parameter).
// Each wave takes its own tiles; the main loop takes them two at a time when
// both lie wholly inside the gradient and issues the next pair's eight 16-byte
// nontemporal loads per lane before encoding the current pair.  The tail takes single tiles with
// bounds-checked 4-byte loads (also used throughout when x is not dword
// aligned, which the interface excludes).
template <typename T, int MODE, bool BL, bool STAGED>
__global__ __launch_bounds__(kBlock) void encode_dense_kernel(
    const T* __restrict__ x, T* __restrict__ y, uint32_t* __restrict__ b, uint64_t n,
    uint64_t words, uint64_t seed, uint32_t rows, uint32_t block, uint32_t c, uint32_t cmask,
    uint32_t log2c, bool vec, uint32_t bk, uint32_t brows, StageOut so) {
    typedef typename Vec4<T>::type V;
    __shared__ uint2 s_stage[STAGED ? kBlock : 1];  // staged: kStageCap entries per wave
    uint2* const stage = s_stage + (STAGED ? (threadIdx.x & ~63u) : 0u);
    const uint32_t lane = lane_id();
    const uint64_t gwave = (uint64_t)blockIdx.x * (kBlock / 64) + uniform(threadIdx.x >> 6);
    const uint64_t nwaves = (uint64_t)gridDim.x * (kBlock / 64);
    const uint64_t ntiles = (n + kTile - 1) / kTile;
    const uint64_t npairs = vec ? n / (2 * kTile) : 0;

    // a buffer resource over the pair's 8 KiB, built on the scalar unit: the
    // lanes' offsets never change, so no per-pair vector address arithmetic
    // competes for the registers that the loads in flight hold
    auto load_pair = [&](uint64_t q, V (&v)[8]) {
        const __amdgpu_buffer_rsrc_t rs =
            buffer_rsrc(x + q * (2 * kTile), (uint32_t)(2 * kTile * sizeof(T)));
#pragma unroll
        for (int u = 0; u < 8; u++) v[u] = buffer_load16_nt<V>(rs, 16u * lane, 1024u * u);
    };
    auto encode_pair = [&](uint64_t q, const V (&v)[8]) {
#pragma unroll
        for (int h = 0; h < 2; h++) {
            T e[4][4];
#pragma unroll
            for (int l = 0; l < 4; l++) {
                e[l][0] = v[4 * h + l].x;
                e[l][1] = v[4 * h + l].y;
                e[l][2] = v[4 * h + l].z;
                e[l][3] = v[4 * h + l].w;
            }
            encode_tile<T, MODE, BL, STAGED>(e, (2 * q + h) * kTile, lane, y, b, words, seed, rows,
                                             block, c, cmask, log2c, bk, brows, so, stage);
        }
    };
    // rolling pipeline: the next pair's loads are issued before the current
    // pair is encoded (never conditionally on their own, so the compiler's
    // load waits leave exactly them in flight)
    uint64_t q = gwave;
    if (q < npairs) {
        V va[8], vb[8];
        load_pair(q, va);
        for (;;) {
            if (q + nwaves >= npairs) {
                encode_pair(q, va);
                break;
            }
            load_pair(q + nwaves, vb);
            encode_pair(q, va);
            q += nwaves;
            if (q + nwaves >= npairs) {
                encode_pair(q, vb);
                break;
            }
            load_pair(q + nwaves, va);
            encode_pair(q, vb);
            q += nwaves;
        }
    }
    for (uint64_t tile = 2 * npairs + gwave; tile < ntiles; tile += nwaves) {
        const uint64_t tbase = tile * kTile;
        T e[4][4];
#pragma unroll
        for (int l = 0; l < 4; l++)
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const uint64_t p = tbase + 256ull * l + 4ull * lane + k;
                e[l][k] = p < n ? x[p] : T(0);
            }
        encode_tile<T, MODE, BL, STAGED>(e, tbase, lane, y, b, words, seed, rows, block, c, cmask,
                                         log2c, bk, brows, so, stage);
    }
}

template <typename T>
__global__ __launch_bounds__(kBlock) void encode_coo_kernel(
    const uint32_t* __restrict__ idx, const T* __restrict__ val, uint64_t nnz,
    T* __restrict__ y, uint32_t* __restrict__ b, uint64_t n, uint64_t seed, uint32_t brows,
    uint32_t block, uint32_t c, uint32_t cmask, uint32_t log2c, uint32_t bk,
    uint32_t bloom_rows) {
    const uint64_t stride = (uint64_t)gridDim.x * kBlock;
    for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < nnz; i += stride) {
        const uint32_t p = idx[i];
        const T v = val[i];
        if (p >= n || !Val<T>::nonzero(v)) continue;
        if (bk == 0u)
            atomicOr(b + (p >> 5), 1u << (p & 31u));
        else
            bloom_insert_param(b, p, seed, bk, bloom_rows, c, cmask, log2c);
        const BatchHash h =
            batch_hash_blocked(seed, brows, cmask, log2c, (uint64_t)(p >> log2c), block);
        const uint32_t t = p & cmask;
#pragma unroll
        for (int j = 0; j < 3; j++)
            Val<T>::atomic_add(y + cell_of(h, j, t, c, cmask), Val<T>::sign(v, (h.neg >> j) & 1u));
    }
}

uint32_t grid_for(uint64_t work_items, uint64_t per_block, uint32_t cap) {
    uint64_t g = (work_items + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (uint32_t)g;
}

template <typename T, int MODE, bool BL, bool STAGED = false>
hipError_t launch_dense_t(const Geo& g, const void* x, void* y, uint32_t* b, hipStream_t s,
                          uint64_t ntiles, int cus, StageOut so = StageOut{nullptr, nullptr, 0}) {
    // the workgroups that are resident at once stride over the tiles; when
    // that leaves each wave fewer than 64 tiles, four times as many, so the
    // dispatcher evens out the last ones (measured on MI355X: VGG19- and
    // BERT-base-sized gradients 4 % faster; at 2^30 parameters no change)
    int per_cu = 0;  // resident workgroups per CU
    const hipError_t e = occupancy_per_cu(
        reinterpret_cast<const void*>(&encode_dense_kernel<T, MODE, BL, STAGED>), kBlock, &per_cu);
    if (e != hipSuccess) return e;
    const uint64_t resident = (uint64_t)cus * per_cu;
    const uint64_t mult = ntiles < 64 * resident * (kBlock / 64) ? 4 : 1;
    const uint32_t grid = grid_for(ntiles, 2 * (kBlock / 64), (uint32_t)(resident * mult));
    hipLaunchKernelGGL((encode_dense_kernel<T, MODE, BL, STAGED>), dim3(grid), dim3(kBlock), 0, s,
                       static_cast<const T*>(x), static_cast<T*>(y), b, g.n, g.words, g.seed,
                       g.brows, g.block, g.c, g.cmask, g.log2c,
                       // a dword-aligned gradient (every valid one) takes the
                       // 16-byte buffer loads, also off the 16-byte grid: a
                       // view 8 bytes off it took the element-wise loads, 1.5 x
                       // the time
                       (reinterpret_cast<uintptr_t>(x) & 3u) == 0, g.bloom_k, g.bloom_rows, so);
    return hipGetLastError();
}


// ---- gathered encode (through the plan) ------------------------------------------
//
// One workgroup per sketch row (grid-stride) assembles the row in LDS from the
// plan's list of (batch, hash) pairs landing on it: each wave takes one pair at
// a time, reads the batch's c values (coalesced 16-byte loads, C/256 per lane)
// and adds g_j * x_t into cell (t + bias_j) mod c of the row.  Within one pair
// the cells are a rotation, so the LDS adds of a wave never collide.  int32
// waves add into one copy of the row with LDS atomics; fp32 waves each keep a
// copy of their own, added to without atomics (LDS float atomics measured
// about five times slower than integer ones here) and summed in wave order at
// the end, so the fp32 sums are also reproducible.  The
// pair with j = 0 of each batch (there is exactly one) also writes the batch's
// bitmap words, all of them, from the same loads.  Every batch is read once per
// hash, 12n bytes in all whatever the density, and no global atomics are used.
template <typename T>
struct GatherArgs {
    const PlanHeader* hdr;
    const uint32_t* rowoff;
    const uint2* entry;
    const T* x;
    T* y;
    uint32_t* b;
    uint64_t n, seed, words;
    uint32_t rows;
    bool vec;  // x is 16-byte aligned
};

template <typename T, int C>
__global__ __launch_bounds__(kBlock) void encode_gather_kernel(GatherArgs<T> a) {
    typedef typename Vec4<T>::type V;
    constexpr uint32_t NV = C / 256;  // 16-byte loads per lane per batch
    constexpr uint32_t WPB = C / 32;  // bitmap words per batch
    constexpr uint32_t kWaves = kBlock / 64;
    constexpr bool kPrivate = std::is_same<T, float>::value;  // one copy of the row per wave
    constexpr uint32_t kCopies = kPrivate ? kWaves : 1u;
    __shared__ T s_acc[kCopies * C];
    const PlanHeader* hdr = a.hdr;
    const bool ok = hdr->magic == kPlanMagic && hdr->n == a.n && hdr->seed == a.seed &&
                    hdr->c == (uint32_t)C && hdr->rows == a.rows;
    if (!ok) {
        // a plan of another geometry: a zero sketch and an all-ones bitmap,
        // which no decode can mistake for a gradient
        const uint64_t stride = (uint64_t)gridDim.x * kBlock;
        const uint64_t cells = (uint64_t)a.rows * C;
        for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < cells; i += stride)
            a.y[i] = T(0);
        for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < a.words; i += stride)
            a.b[i] = 0xffffffffu;
        return;
    }
    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    for (uint32_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
        for (uint32_t k = threadIdx.x; k < kCopies * C; k += kBlock) s_acc[k] = T(0);
        lds_barrier();
        T* const mine = s_acc + (kPrivate ? wave * C : 0u);
        const uint32_t e0 = a.rowoff[row], e1 = a.rowoff[row + 1];
        for (uint32_t e = e0 + wave; e < e1; e += kWaves) {
            const uint2 ent = a.entry[e];
            const uint32_t bias = ent.y & 0xffffu, j = (ent.y >> 16) & 3u;
            const bool neg = (ent.y >> 31) != 0u;
            const uint64_t base = (uint64_t)ent.x * C;
            // value t = 256 u + 4 lane + k of the batch is v[u][k]
            T v[NV][4];
            if (a.vec && base + C <= a.n) {
                const V* src = reinterpret_cast<const V*>(a.x + base) + lane;
#pragma unroll
                for (uint32_t u = 0; u < NV; u++) {
                    const V q = __builtin_nontemporal_load(src + 64 * u);
                    v[u][0] = q.x;
                    v[u][1] = q.y;
                    v[u][2] = q.z;
                    v[u][3] = q.w;
                }
            } else {
#pragma unroll
                for (uint32_t u = 0; u < NV; u++)
#pragma unroll
                    for (uint32_t k = 0; k < 4; k++) {
                        const uint64_t p = base + 256u * u + 4u * lane + k;
                        v[u][k] = p < a.n ? a.x[p] : T(0);
                    }
            }
            if (j == 0u) {
                // word w of the batch holds t = 32 w .. 32 w + 31: lanes
                // 8 (w mod 8) .. + 7 of load w / 8, parameter 4 lane' + k at
                // bit 4 (lane' - 8 (w mod 8)) + k
                uint64_t m[NV][4];
#pragma unroll
                for (uint32_t u = 0; u < NV; u++)
#pragma unroll
                    for (uint32_t k = 0; k < 4; k++) m[u][k] = __ballot(Val<T>::nonzero(v[u][k]));
                if (lane < WPB) {
                    const uint32_t u = lane >> 3, sh = 8u * (lane & 7u);
                    uint32_t word = 0;
#pragma unroll
                    for (uint32_t k = 0; k < 4; k++) {
                        uint64_t mk = m[0][k];
#pragma unroll
                        for (uint32_t uu = 1; uu < NV; uu++)
                            if (u == uu) mk = m[uu][k];
                        word |= spread4((uint32_t)(mk >> sh)) << k;
                    }
                    const uint64_t widx = (uint64_t)ent.x * WPB + lane;
                    if (widx < a.words) a.b[widx] = word;
                }
            }
#pragma unroll
            for (uint32_t u = 0; u < NV; u++)
#pragma unroll
                for (uint32_t k = 0; k < 4; k++) {
                    if (!Val<T>::nonzero(v[u][k])) continue;
                    const uint32_t t = 256u * u + 4u * lane + k;
                    const T add = Val<T>::sign(v[u][k], neg);
                    const uint32_t cell = (t + bias) & (uint32_t)(C - 1);
                    if (kPrivate)
                        mine[cell] += add;
                    else
                        atomicAdd(&mine[cell], add);
                }
        }
        lds_barrier();
        T* dst = a.y + (uint64_t)row * C;
        for (uint32_t k = threadIdx.x; k < (uint32_t)C; k += kBlock) {
            T acc = s_acc[k];
#pragma unroll
            for (uint32_t w = 1; w < kCopies; w++) acc += s_acc[w * C + k];
            dst[k] = acc;
        }
        lds_barrier();  // the copies are cleared for the next row
    }
}

template <typename T, int C>
hipError_t launch_gather_t(const Geo& g, const void* plan, const void* x, void* y, uint32_t* b,
                           hipStream_t s, int cus) {
    const PlanLayout L = plan_layout(g);
    const char* base = static_cast<const char*>(plan);
    GatherArgs<T> a;
    a.hdr = reinterpret_cast<const PlanHeader*>(base + L.header);
    a.rowoff = reinterpret_cast<const uint32_t*>(base + L.rowoff);
    a.entry = reinterpret_cast<const uint2*>(base + L.entry);
    a.x = static_cast<const T*>(x);
    a.y = static_cast<T*>(y);
    a.b = b;
    a.n = g.n;
    a.seed = g.seed;
    a.words = g.words;
    a.rows = g.rows;
    a.vec = (reinterpret_cast<uintptr_t>(x) & 15u) == 0;
    const uint32_t grid = g.rows < (uint32_t)cus * 8 ? g.rows : (uint32_t)cus * 8;
    hipLaunchKernelGGL((encode_gather_kernel<T, C>), dim3(grid), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

// ---- staged encode, second pass: rows from the staged lists ----------------------
//
// One wave per sketch row (grid-stride) sums the row in its own LDS copy: for
// every (batch, hash j) pair of the row's plan entries, g_j * value into cell
// (t + bias_j) mod C for each nonzero (t, value) of the batch -- taken from the
// batch's staged list when the list holds them all, else from the gradient
// itself (the batch's C values, coalesced, as in the gathered encode).  The
// entries are taken 64 at a time, one per lane, which loads it and its
// batch's count; a wave prefix sum gives each listed nonzero a slot, and the
// lanes take slots in turn with kAhead list loads in flight each.  Batches
// past the list capacity go one at a time.  Within one pair the cells are a
// rotation and never collide; different pairs of a row may, so the adds are
// LDS atomics (int32 wraps; fp32 sums in an unspecified order, like
// hc_encode's global atomics).  The row is then stored once, so the sketch
// needs no clearing and takes no global atomics.  A wave per row, with no
// workgroup barriers, keeps four times as many rows in flight as a workgroup
// per row: a row is a few dependent memory latencies whatever its size.
template <typename T>
struct RowsArgs {
    const PlanHeader* hdr;
    const uint32_t* rowoff;
    const uint2* entry;
    const uint32_t* count;
    const uint2* list;
    const T* x;
    T* y;
    uint32_t* b;
    uint64_t n, seed, words, nb;
    uint32_t rows;
    bool vec;    // x is 16-byte aligned
    bool y_vec;  // y is 16-byte aligned
};

template <typename T>
__device__ __forceinline__ T bits_value(uint32_t v) {
    return __builtin_bit_cast(T, v);
}

template <typename T>
__device__ __forceinline__ void lds_add(T* a, T v) {
    if constexpr (std::is_same<T, int32_t>::value)
        atomicAdd(reinterpret_cast<unsigned int*>(a), (unsigned int)v);
    else
        atomicAdd(a, v);
}

template <typename T, int C>
__global__ __launch_bounds__(kBlock) void stage_rows_kernel(RowsArgs<T> a) {
    typedef typename Vec4<T>::type V;
    constexpr uint32_t NV = C / 256;  // 16-byte vectors per lane per row (and per batch)
    constexpr uint32_t kWaves = kBlock / 64;
    constexpr uint32_t kAhead = 4;    // listed nonzeros per lane with loads in flight
    __shared__ __align__(16) T s_rows[kWaves * C];
    const PlanHeader* hdr = a.hdr;
    const bool ok = hdr->magic == kPlanMagic && hdr->n == a.n && hdr->seed == a.seed &&
                    hdr->c == (uint32_t)C && hdr->rows == a.rows;
    if (!ok) {
        // a plan of another geometry: a zero sketch and an all-ones bitmap,
        // which no decode can mistake for a gradient
        const uint64_t stride = (uint64_t)gridDim.x * kBlock;
        const uint64_t cells = (uint64_t)a.rows * C;
        for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < cells; i += stride)
            a.y[i] = T(0);
        for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < a.words; i += stride)
            a.b[i] = 0xffffffffu;
        return;
    }
    const uint32_t lane = lane_id();
    const uint32_t wave = uniform(threadIdx.x >> 6);
    T* const acc = s_rows + wave * C;
    const uint32_t nwaves = gridDim.x * kWaves;
    for (uint32_t row = blockIdx.x * kWaves + wave; row < a.rows; row += nwaves) {
        // a wave's LDS operations complete in order: the previous row's reads
        // are done before these stores
#pragma unroll
        for (uint32_t q = 0; q < NV; q++) {
            const V z = {T(0), T(0), T(0), T(0)};
            *reinterpret_cast<V*>(acc + 256u * q + 4u * lane) = z;
        }
        const uint32_t e0 = a.rowoff[row], e1 = a.rowoff[row + 1];
        for (uint32_t cb = e0; cb < e1; cb += 64u) {
            const uint32_t e = cb + lane;
            uint2 ent = make_uint2(0u, 0u);
            uint32_t m = 0;
            if (e < e1) {
                ent = a.entry[e];
                if (ent.x < a.nb) m = a.count[ent.x];
            }
            const uint32_t lm = m <= kStageCap ? m : 0u;  // listed nonzeros of this lane's pair
            uint32_t incl = lm;
#pragma unroll
            for (uint32_t d = 1; d < 64; d <<= 1) {
                const uint32_t y = __shfl_up(incl, d);
                if (lane >= d) incl += y;
            }
            const uint32_t total = __shfl(incl, 63);
            for (uint32_t i0 = 0; i0 < total; i0 += 64u * kAhead) {
                uint2 it[kAhead];
                uint32_t eb[kAhead];
#pragma unroll
                for (uint32_t u = 0; u < kAhead; u++) {
                    // slot i belongs to the first lane whose inclusive sum
                    // exceeds it (every lane searches, so the shuffles see
                    // the whole wave)
                    const uint32_t i = i0 + 64u * u + lane;
                    const uint32_t ic = i < total ? i : total - 1u;
                    uint32_t pos = 0;
#pragma unroll
                    for (uint32_t step = 32; step >= 1; step >>= 1)
                        if ((uint32_t)__shfl(incl, (int)(pos + step - 1u)) <= ic) pos += step;
                    const uint32_t first = (uint32_t)__shfl(incl, (int)pos) -
                                           (uint32_t)__shfl(lm, (int)pos);
                    const uint32_t bx = (uint32_t)__shfl(ent.x, (int)pos);
                    eb[u] = (uint32_t)__shfl(ent.y, (int)pos);
                    it[u] = make_uint2(0u, 0u);
                    if (i < total) it[u] = a.list[(uint64_t)bx * kStageCap + (ic - first)];
                }
#pragma unroll
                for (uint32_t u = 0; u < kAhead; u++) {
                    if (i0 + 64u * u + lane >= total) continue;
                    const uint32_t cell = (it[u].x + (eb[u] & 0xffffu)) & (uint32_t)(C - 1);
                    lds_add(&acc[cell], Val<T>::sign(bits_value<T>(it[u].y), (eb[u] >> 31) != 0u));
                }
            }
            // batches past the list capacity: the batch's values from x
            uint64_t big = __ballot(m > kStageCap);
            while (big != 0ull) {
                const uint32_t src = (uint32_t)__ffsll((unsigned long long)big) - 1u;
                big &= big - 1ull;
                const uint32_t bx = (uint32_t)__shfl(ent.x, (int)src);
                const uint32_t ey = (uint32_t)__shfl(ent.y, (int)src);
                const uint32_t bias = ey & 0xffffu;
                const bool neg = (ey >> 31) != 0u;
                const uint64_t bbase = (uint64_t)bx * C;
                T v[NV][4];
                if (a.vec && bbase + C <= a.n) {
                    const V* src4 = reinterpret_cast<const V*>(a.x + bbase) + lane;
#pragma unroll
                    for (uint32_t u = 0; u < NV; u++) {
                        const V q = __builtin_nontemporal_load(src4 + 64 * u);
                        v[u][0] = q.x;
                        v[u][1] = q.y;
                        v[u][2] = q.z;
                        v[u][3] = q.w;
                    }
                } else {
#pragma unroll
                    for (uint32_t u = 0; u < NV; u++)
#pragma unroll
                        for (uint32_t k = 0; k < 4; k++) {
                            const uint64_t p = bbase + 256u * u + 4u * lane + k;
                            v[u][k] = p < a.n ? a.x[p] : T(0);
                        }
                }
#pragma unroll
                for (uint32_t u = 0; u < NV; u++)
#pragma unroll
                    for (uint32_t k = 0; k < 4; k++) {
                        if (!Val<T>::nonzero(v[u][k])) continue;
                        const uint32_t t = 256u * u + 4u * lane + k;
                        lds_add(&acc[(t + bias) & (uint32_t)(C - 1)], Val<T>::sign(v[u][k], neg));
                    }
            }
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // every lane's LDS adds have landed
        __builtin_amdgcn_wave_barrier();
        T* dst = a.y + (uint64_t)row * C;
        if (a.y_vec) {
#pragma unroll
            for (uint32_t q = 0; q < NV; q++)
                reinterpret_cast<V*>(dst)[64u * q + lane] =
                    *reinterpret_cast<const V*>(acc + 256u * q + 4u * lane);
        } else {
#pragma unroll
            for (uint32_t q = 0; q < 4 * NV; q++) dst[64u * q + lane] = acc[64u * q + lane];
        }
    }
}

template <typename T, int C>
hipError_t launch_stage_rows_t(const Geo& g, const void* plan, const StageLayout& SL, void* ws,
                               const void* x, void* y, uint32_t* b, hipStream_t s, int cus) {
    const PlanLayout L = plan_layout(g);
    const char* pb = static_cast<const char*>(plan);
    char* wb = static_cast<char*>(ws);
    RowsArgs<T> a;
    a.hdr = reinterpret_cast<const PlanHeader*>(pb + L.header);
    a.rowoff = reinterpret_cast<const uint32_t*>(pb + L.rowoff);
    a.entry = reinterpret_cast<const uint2*>(pb + L.entry);
    a.count = reinterpret_cast<const uint32_t*>(wb + SL.count);
    a.list = reinterpret_cast<const uint2*>(wb + SL.list);
    a.x = static_cast<const T*>(x);
    a.y = static_cast<T*>(y);
    a.b = b;
    a.n = g.n;
    a.seed = g.seed;
    a.words = g.bwords;
    a.nb = SL.nb;
    a.rows = g.rows;
    a.vec = (reinterpret_cast<uintptr_t>(x) & 15u) == 0;
    a.y_vec = (reinterpret_cast<uintptr_t>(y) & 15u) == 0;
    // one wave per row, four per workgroup, every row in flight at once when
    // the chip holds that many workgroups
    int per_cu = 0;
    hipError_t e = occupancy_per_cu(reinterpret_cast<const void*>(&stage_rows_kernel<T, C>), kBlock,
                                    &per_cu);
    if (e != hipSuccess) return e;
    const uint64_t want = ((uint64_t)g.rows + kBlock / 64 - 1) / (kBlock / 64);
    const uint64_t cap = (uint64_t)cus * per_cu;
    const uint32_t grid = (uint32_t)(want < cap ? want : cap);
    hipLaunchKernelGGL((stage_rows_kernel<T, C>), dim3(grid), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

template <typename T, bool BL>
hipError_t launch_staged_t(const Geo& g, const void* plan, void* ws, const void* x, void* y,
                           uint32_t* b, hipStream_t s, int cus) {
    const StageLayout SL = stage_layout(g);
    char* wb = static_cast<char*>(ws);
    StageOut so;
    so.list = reinterpret_cast<uint2*>(wb + SL.list);
    so.count = reinterpret_cast<uint32_t*>(wb + SL.count);
    so.nb = SL.nb;
    const uint64_t ntiles = (g.n + kTile - 1) / kTile;
    hipError_t e = launch_dense_t<T, 0, BL, true>(g, x, y, b, s, ntiles, cus, so);
    if (e != hipSuccess) return e;
    if (g.c == 1024) return launch_stage_rows_t<T, 1024>(g, plan, SL, ws, x, y, b, s, cus);
    if (g.c == 512) return launch_stage_rows_t<T, 512>(g, plan, SL, ws, x, y, b, s, cus);
    return launch_stage_rows_t<T, 256>(g, plan, SL, ws, x, y, b, s, cus);
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

}  // namespace

StageLayout stage_layout(const Geo& g) {
    StageLayout L;
    L.nb = (g.n + g.c - 1) / g.c;
    size_t o = 0;
    L.count = o;  o = align256(o + L.nb * 4);
    L.list = o;   o = align256(o + L.nb * kStageCap * 8);
    L.total = o;
    return L;
}

hipError_t launch_encode_staged(const Geo& g, const void* plan, void* ws, const void* x, void* y,
                                uint32_t* b, hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    // nothing is cleared: the first pass writes every bitmap word and every
    // batch count, the second every sketch cell; a Bloom filter, which the
    // first pass ORs into, is cleared
    if (g.bloom_k != 0) {
        e = launch_fill_u32(b, g.bwords, 0u, s);
        if (e != hipSuccess) return e;
        if (g.f32) return launch_staged_t<float, true>(g, plan, ws, x, y, b, s, di.cus);
        return launch_staged_t<int32_t, true>(g, plan, ws, x, y, b, s, di.cus);
    }
    if (g.f32) return launch_staged_t<float, false>(g, plan, ws, x, y, b, s, di.cus);
    return launch_staged_t<int32_t, false>(g, plan, ws, x, y, b, s, di.cus);
}

hipError_t launch_fill2_u32(uint32_t* p, uint64_t count, uint32_t* p2, uint64_t count2,
                            uint32_t value, hipStream_t s) {
    if (count == 0 && count2 == 0) return hipSuccess;
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    // one workgroup per kFillVecs vectors of an aligned range; an unaligned
    // one is grid-strided over workgroups in proportion to its size
    const bool vec = (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
    const bool vec2 = (reinterpret_cast<uintptr_t>(p2) & 15u) == 0;
    const uint32_t cap = (uint32_t)di.cus * 16;
    auto groups = [&](uint64_t cnt, bool v) -> uint32_t {
        if (cnt == 0) return 0u;
        if (!v) return grid_for(cnt, kBlock, cap);
        const uint64_t g = (cnt / 4 + kFillVecs - 1) / kFillVecs;
        return g == 0 ? 1u : (uint32_t)g;
    };
    const uint32_t g0 = groups(count, vec);
    const uint32_t g1 = groups(count2, vec2);
    hipLaunchKernelGGL(fill_u32_kernel, dim3(g0 + g1), dim3(kBlock), 0, s, p, count, vec, p2,
                       count2, vec2, g0, value);
    return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, uint64_t count, uint32_t value, hipStream_t s) {
    return launch_fill2_u32(p, count, nullptr, 0, value, s);
}

hipError_t launch_encode_dense(const Geo& g, const void* x, void* y, uint32_t* b,
                               hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    // the sketch and the index start from zero: the kernel adds into the
    // sketch, stores only the bitmap's nonzero words, and ORs into a filter
    e = launch_fill2_u32(static_cast<uint32_t*>(y), g.cells, b, g.bwords, 0u, s);
    if (e != hipSuccess) return e;
    const uint64_t ntiles = (g.n + kTile - 1) / kTile;
    const int mode = g.c >= 256 ? 0 : (g.c >= 4 ? 1 : 2);
    if (g.bloom_k != 0) {
        if (g.f32) {
            if (mode == 0) return launch_dense_t<float, 0, true>(g, x, y, b, s, ntiles, di.cus);
            if (mode == 1) return launch_dense_t<float, 1, true>(g, x, y, b, s, ntiles, di.cus);
            return launch_dense_t<float, 2, true>(g, x, y, b, s, ntiles, di.cus);
        }
        if (mode == 0) return launch_dense_t<int32_t, 0, true>(g, x, y, b, s, ntiles, di.cus);
        if (mode == 1) return launch_dense_t<int32_t, 1, true>(g, x, y, b, s, ntiles, di.cus);
        return launch_dense_t<int32_t, 2, true>(g, x, y, b, s, ntiles, di.cus);
    }
    if (g.f32) {
        if (mode == 0) return launch_dense_t<float, 0, false>(g, x, y, b, s, ntiles, di.cus);
        if (mode == 1) return launch_dense_t<float, 1, false>(g, x, y, b, s, ntiles, di.cus);
        return launch_dense_t<float, 2, false>(g, x, y, b, s, ntiles, di.cus);
    }
    if (mode == 0) return launch_dense_t<int32_t, 0, false>(g, x, y, b, s, ntiles, di.cus);
    if (mode == 1) return launch_dense_t<int32_t, 1, false>(g, x, y, b, s, ntiles, di.cus);
    return launch_dense_t<int32_t, 2, false>(g, x, y, b, s, ntiles, di.cus);
}


hipError_t launch_encode_gather(const Geo& g, const void* plan, const void* x, void* y,
                                uint32_t* b, hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    if (g.f32) {
        if (g.c == 1024) return launch_gather_t<float, 1024>(g, plan, x, y, b, s, di.cus);
        if (g.c == 512) return launch_gather_t<float, 512>(g, plan, x, y, b, s, di.cus);
        return launch_gather_t<float, 256>(g, plan, x, y, b, s, di.cus);
    }
    if (g.c == 1024) return launch_gather_t<int32_t, 1024>(g, plan, x, y, b, s, di.cus);
    if (g.c == 512) return launch_gather_t<int32_t, 512>(g, plan, x, y, b, s, di.cus);
    return launch_gather_t<int32_t, 256>(g, plan, x, y, b, s, di.cus);
}

hipError_t launch_encode_coo(const Geo& g, const uint32_t* idx, const void* val, uint64_t nnz,
                             void* y, uint32_t* b, hipStream_t s) {
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;
    e = launch_fill2_u32(static_cast<uint32_t*>(y), g.cells, b, g.bwords, 0u, s);
    if (e != hipSuccess) return e;
    if (nnz == 0) return hipSuccess;
    const uint32_t grid = grid_for(nnz, kBlock, (uint32_t)di.cus * 16);
    if (g.f32)
        hipLaunchKernelGGL(encode_coo_kernel<float>, dim3(grid), dim3(kBlock), 0, s, idx,
                           static_cast<const float*>(val), nnz, static_cast<float*>(y), b, g.n,
                           g.seed, g.brows, g.block, g.c, g.cmask, g.log2c, g.bloom_k,
                           g.bloom_rows);
    else
        hipLaunchKernelGGL(encode_coo_kernel<int32_t>, dim3(grid), dim3(kBlock), 0, s, idx,
                           static_cast<const int32_t*>(val), nnz, static_cast<int32_t*>(y), b,
                           g.n, g.seed, g.brows, g.block, g.c, g.cmask, g.log2c, g.bloom_k,
                           g.bloom_rows);
    return hipGetLastError();
}

}  // namespace hc
