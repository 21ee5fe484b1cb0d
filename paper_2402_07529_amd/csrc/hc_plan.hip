// hc_plan.hip -- the inverse row map of a sketch geometry.
//
// Under section 3.4's batching every batch b of c parameters lands, for each
// hash j, on one whole sketch row r_j(b), rotated by bias_j(b).  The plan lists,
// for every row, the (batch, j) pairs that land on it, so a workgroup that owns
// a row can gather everything that falls into it instead of receiving
// scattered atomics.  It depends only on (n, c, rows, seed), so one plan serves
// every worker and every iteration of a training run.
//
// Layout (device memory, offsets from the plan base, all 256-byte aligned):
//   PlanHeader                 geometry it was built for
//   rowoff[rows + 1]  uint32   exclusive offsets of each row's entries
//   entry[3 * nb]     uint2    .x = batch, .y = bias | j << 16 | (g_j < 0) << 31
//   scratch[...]               block sums of the scan, row cursors (build only)
#include "hc_device.h"
#include "hc_internal.h"

namespace hc {

namespace {

constexpr int kBlock = 256;
constexpr uint32_t kScanItems = 16;                       // per lane
constexpr uint32_t kScanTile = kBlock * kScanItems;      // per workgroup

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

__global__ void plan_header_kernel(PlanHeader* h, uint64_t n, uint64_t seed, uint32_t c,
                                   uint32_t rows) {
    if (threadIdx.x == 0) {
        h->n = n;
        h->seed = seed;
        h->c = c;
        h->rows = rows;
        h->magic = kPlanMagic;
        h->pad = 0;
    }
}

__global__ __launch_bounds__(kBlock) void plan_count_kernel(uint32_t* __restrict__ rowcnt,
                                                            uint64_t nb, uint64_t seed,
                                                            uint32_t rows, uint32_t cmask) {
    const uint64_t step = (uint64_t)gridDim.x * kBlock;
    for (uint64_t b = (uint64_t)blockIdx.x * kBlock + threadIdx.x; b < nb; b += step) {
        const BatchHash h = batch_hash(seed, rows, cmask, b);
#pragma unroll
        for (int j = 0; j < 3; j++) atomicAdd(rowcnt + h.row[j], 1u);
    }
}

// Three-pass exclusive scan of a uint32 array (sums fit in 32 bits).
__global__ __launch_bounds__(kBlock) void scan_tiles_kernel(const uint32_t* __restrict__ in,
                                                            uint64_t len,
                                                            uint32_t* __restrict__ tile_sum) {
    __shared__ uint32_t s_tmp[kBlock / 64];
    const uint64_t base = (uint64_t)blockIdx.x * kScanTile + (uint64_t)threadIdx.x * kScanItems;
    uint32_t s = 0;
    for (uint32_t i = 0; i < kScanItems; i++)
        if (base + i < len) s += in[base + i];
    uint32_t total;
    block_exclusive_scan(s, s_tmp, &total);
    if (threadIdx.x == 0) tile_sum[blockIdx.x] = total;
}

// One workgroup: exclusive scan of the tile sums in place; out_total gets the sum.
__global__ __launch_bounds__(1024) void scan_tile_sums_kernel(uint32_t* __restrict__ tile_sum,
                                                              uint64_t ntiles,
                                                              uint32_t* __restrict__ out_total) {
    __shared__ uint32_t s_tmp[16];
    const uint64_t per = (ntiles + 1023) / 1024;
    const uint64_t lo = (uint64_t)threadIdx.x * per;
    const uint64_t hi = lo + per < ntiles ? lo + per : ntiles;
    uint32_t s = 0;
    for (uint64_t i = lo; i < hi; i++) s += tile_sum[i];
    uint32_t total;
    uint32_t off = block_exclusive_scan(s, s_tmp, &total);
    for (uint64_t i = lo; i < hi; i++) {
        const uint32_t v = tile_sum[i];
        tile_sum[i] = off;
        off += v;
    }
    if (threadIdx.x == 0) *out_total = total;
}

// out[i] = exclusive prefix of in; also copies it to cursor (if non-null).
__global__ __launch_bounds__(kBlock) void scan_write_kernel(const uint32_t* __restrict__ in,
                                                            uint64_t len,
                                                            const uint32_t* __restrict__ tile_sum,
                                                            uint32_t* __restrict__ out,
                                                            uint32_t* __restrict__ cursor) {
    __shared__ uint32_t s_tmp[kBlock / 64];
    const uint64_t base = (uint64_t)blockIdx.x * kScanTile + (uint64_t)threadIdx.x * kScanItems;
    uint32_t v[kScanItems];
    uint32_t s = 0;
    for (uint32_t i = 0; i < kScanItems; i++) {
        v[i] = base + i < len ? in[base + i] : 0u;
        s += v[i];
    }
    uint32_t total;
    uint32_t off = tile_sum[blockIdx.x] + block_exclusive_scan(s, s_tmp, &total);
    for (uint32_t i = 0; i < kScanItems; i++) {
        if (base + i < len) {
            out[base + i] = off;
            if (cursor) cursor[base + i] = off;
        }
        off += v[i];
    }
}

__global__ __launch_bounds__(kBlock) void plan_fill_kernel(uint32_t* __restrict__ cursor,
                                                           uint2* __restrict__ entry, uint64_t nb,
                                                           uint64_t seed, uint32_t rows,
                                                           uint32_t cmask) {
    const uint64_t step = (uint64_t)gridDim.x * kBlock;
    for (uint64_t b = (uint64_t)blockIdx.x * kBlock + threadIdx.x; b < nb; b += step) {
        const BatchHash h = batch_hash(seed, rows, cmask, b);
#pragma unroll
        for (int j = 0; j < 3; j++) {
            const uint32_t slot = atomicAdd(cursor + h.row[j], 1u);
            entry[slot] = make_uint2((uint32_t)b, h.bias[j] | ((uint32_t)j << 16) |
                                                      (((h.neg >> j) & 1u) << 31));
        }
    }
}

}  // namespace

PlanLayout plan_layout(const Geo& g) {
    PlanLayout L;
    L.nb = (g.n + g.c - 1) / g.c;
    L.ntiles = ((uint64_t)g.rows + kScanTile - 1) / kScanTile;
    size_t o = 0;
    L.header = o;   o = align256(o + sizeof(PlanHeader));
    L.rowoff = o;   o = align256(o + ((size_t)g.rows + 1) * 4);
    L.entry = o;    o = align256(o + (size_t)L.nb * 3 * 8);
    L.rowcnt = o;   o = align256(o + (size_t)g.rows * 4);
    L.tiles = o;    o = align256(o + (size_t)L.ntiles * 4);
    L.total = o;
    return L;
}

bool plan_supported(const Geo& g) { return g.c >= 256 && (uint64_t)((g.n + g.c - 1) / g.c) * 3 < 0xffffffffull; }

hipError_t launch_plan_build(const Geo& g, void* plan, hipStream_t s) {
    const PlanLayout L = plan_layout(g);
    char* base = static_cast<char*>(plan);
    uint32_t* rowoff = reinterpret_cast<uint32_t*>(base + L.rowoff);
    uint2* entry = reinterpret_cast<uint2*>(base + L.entry);
    uint32_t* rowcnt = reinterpret_cast<uint32_t*>(base + L.rowcnt);
    uint32_t* tiles = reinterpret_cast<uint32_t*>(base + L.tiles);
    DeviceInfo di;
    hipError_t e = device_info(&di);
    if (e != hipSuccess) return e;

    hipLaunchKernelGGL(plan_header_kernel, dim3(1), dim3(64), 0, s,
                       reinterpret_cast<PlanHeader*>(base + L.header), g.n, g.seed, g.c, g.rows);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_fill_u32(rowcnt, g.rows, 0u, s)) != hipSuccess) return e;
    uint64_t grid = (L.nb + kBlock - 1) / kBlock;
    if (grid > (uint64_t)di.cus * 16) grid = (uint64_t)di.cus * 16;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(plan_count_kernel, dim3((uint32_t)grid), dim3(kBlock), 0, s, rowcnt, L.nb,
                       g.seed, g.rows, g.cmask);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_tiles_kernel, dim3((uint32_t)L.ntiles), dim3(kBlock), 0, s, rowcnt,
                       (uint64_t)g.rows, tiles);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_tile_sums_kernel, dim3(1), dim3(1024), 0, s, tiles, L.ntiles,
                       rowoff + g.rows);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // rowoff = exclusive prefix; rowcnt becomes the fill cursor
    hipLaunchKernelGGL(scan_write_kernel, dim3((uint32_t)L.ntiles), dim3(kBlock), 0, s, rowcnt,
                       (uint64_t)g.rows, tiles, rowoff, rowcnt);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(plan_fill_kernel, dim3((uint32_t)grid), dim3(kBlock), 0, s, rowcnt, entry,
                       L.nb, g.seed, g.rows, g.cmask);
    return hipGetLastError();
}

}  // namespace hc
