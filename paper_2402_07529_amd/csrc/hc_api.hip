// hc_api.hip -- the C ABI of include/hc.h: argument validation, sketch
// geometry, workspace sizing and kernel launches.  Host code only.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <map>
#include <mutex>
#include <string>
#include <tuple>

#include "../../include/hc.h"
#include "hc_internal.h"

namespace hc {

namespace {

thread_local std::string g_last_error;

hc_status fail(hc_status s, const char* msg) {
    g_last_error = msg;
    return s;
}

hc_status fail_hip(hipError_t e, const char* where) {
    g_last_error = std::string(where) + ": " + hipGetErrorString(e);
    return HC_EHIP;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Validate the public params and convert them to the kernels' form.
hc_status to_geo(const hc_params* p, Geo* g) {
    if (p == nullptr) return fail(HC_EINVAL, "params is NULL");
    if (p->k != 3) return fail(HC_EUNSUPPORTED, "only k = 3 hashes are implemented");
    if (p->vtype != HC_I32 && p->vtype != HC_F32) return fail(HC_EINVAL, "unknown vtype");
    if (p->n == 0 || p->n > 0xffffffffull) return fail(HC_EINVAL, "n must be in [1, 2^32 - 1]");
    if (p->c == 0 || p->c > 1024 || (p->c & (p->c - 1)) != 0)
        return fail(HC_EINVAL, "c must be a power of two in [1, 1024]");
    if (p->rows < 3) return fail(HC_EINVAL, "rows must be >= 3");
    if (p->rows > 0xffffffffull / p->c) return fail(HC_EINVAL, "rows * c must be < 2^32");
    g->n = p->n;
    g->words = (p->n + 31) / 32;
    g->rows = (uint32_t)p->rows;
    g->c = p->c;
    g->cmask = p->c - 1;
    g->log2c = 0;
    while ((1u << g->log2c) < p->c) g->log2c++;
    g->cells = (uint32_t)(p->rows * p->c);
    g->seed = p->seed;
    g->f32 = p->vtype == HC_F32;
    g->block = p->block;
    g->brows = g->rows;
    g->nblocks = 1;
    if (p->block != 0) {
        // section 3.2 blocking: whole bitmap words per block, and every block
        // owning the same whole number (>= 3) of rows
        if (((uint64_t)p->block * p->c) % 32 != 0)
            return fail(HC_EINVAL, "block * c must be a multiple of 32");
        const uint64_t batches = (p->n + p->c - 1) / p->c;
        const uint64_t nblocks = (batches + p->block - 1) / p->block;
        if (p->rows % nblocks != 0)
            return fail(HC_EINVAL, "rows must be a multiple of the number of blocks");
        if (p->rows / nblocks < 3) return fail(HC_EINVAL, "every block needs >= 3 rows");
        g->brows = (uint32_t)(p->rows / nblocks);
        g->nblocks = (uint32_t)nblocks;
    }
    if (p->reserved != 0) return fail(HC_EINVAL, "reserved must be 0");
    g->bloom_k = p->bloom_k;
    g->bloom_rows = 0;
    g->bwords = g->words;
    if (p->bloom_k != 0) {
        // section 3.3: a filter of bloom_rows rows of c bits, bit positions < 2^32
        if (p->bloom_k > 64) return fail(HC_EINVAL, "bloom_k must be <= 64");
        if (p->bloom_rows == 0 || p->bloom_rows > 0xffffffffull / p->c)
            return fail(HC_EINVAL, "bloom_rows must be >= 1 with bloom_rows * c < 2^32");
        if (p->block != 0)
            return fail(HC_EUNSUPPORTED, "a Bloom-filter index needs the global sketch");
        g->bloom_rows = (uint32_t)p->bloom_rows;
        g->bwords = (p->bloom_rows * p->c + 31) / 32;
    }
    return HC_OK;
}

// The LDS kernels of a blocked sketch hold one block per workgroup.
hc_status blocked_supported(const Geo& g) {
    if (g.block > kBlockedMaxBatches) return fail(HC_EUNSUPPORTED, "block must be <= 1024 batches");
    if ((uint64_t)g.brows * g.c > 65536) return fail(HC_EUNSUPPORTED, "a block's sketch must have <= 65536 cells");
    // the kernels' own static LDS (barrier reductions) comes on top
    if (blocked_encode_lds(g) + kLdsReserve > kLdsBytes ||
        blocked_decode_lds(g) + kLdsReserve > kLdsBytes)
        return fail(HC_EUNSUPPORTED, "a block's sketch does not fit in one workgroup's LDS");
    return HC_OK;
}

std::mutex g_dev_mu;
std::map<int, int> g_dev_cus;                                        // device -> CUs
std::map<std::tuple<int, const void*, int>, int> g_occupancy;        // -> workgroups per CU
std::map<std::tuple<int, const void*>, int> g_dyn_lds;               // -> dynamic LDS allowed

}  // namespace

hipError_t device_info(DeviceInfo* out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lk(g_dev_mu);
    auto it = g_dev_cus.find(dev);
    if (it == g_dev_cus.end()) {
        int cus = 0;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        it = g_dev_cus.emplace(dev, cus > 0 ? cus : 1).first;
    }
    out->cus = it->second;
    return hipSuccess;
}

hipError_t occupancy_per_cu(const void* kernel, int block, int* out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lk(g_dev_mu);
    const auto key = std::make_tuple(dev, kernel, block);
    auto it = g_occupancy.find(key);
    if (it == g_occupancy.end()) {
        int v = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, kernel, block, 0);
        if (e != hipSuccess) return e;
        if (v < 1) return hipErrorInvalidConfiguration;
        it = g_occupancy.emplace(key, v).first;
    }
    *out = it->second;
    return hipSuccess;
}

hipError_t allow_dynamic_lds(const void* kernel, int bytes) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lk(g_dev_mu);
    const auto key = std::make_tuple(dev, kernel);
    auto it = g_dyn_lds.find(key);
    if (it != g_dyn_lds.end() && it->second >= bytes) return hipSuccess;
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    g_dyn_lds[key] = bytes;
    return hipSuccess;
}

}  // namespace hc

using namespace hc;

extern "C" {

const char* hc_status_string(hc_status s) {
    switch (s) {
        case HC_OK: return "HC_OK";
        case HC_EINVAL: return "HC_EINVAL";
        case HC_EWORKSPACE: return "HC_EWORKSPACE";
        case HC_EHIP: return "HC_EHIP";
        case HC_EUNSUPPORTED: return "HC_EUNSUPPORTED";
    }
    return "HC_UNKNOWN";
}

const char* hc_last_error(void) { return g_last_error.c_str(); }

hc_status hc_geometry(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c, uint64_t seed,
                      hc_vtype vtype, hc_params* out) {
    g_last_error.clear();
    if (out == nullptr) return fail(HC_EINVAL, "out is NULL");
    if (!(gamma > 0.0) || !isfinite(gamma)) return fail(HC_EINVAL, "gamma must be > 0");
    if (c == 0 || c > 1024 || (c & (c - 1)) != 0)
        return fail(HC_EINVAL, "c must be a power of two in [1, 1024]");
    const double need = gamma * (double)n_nonzero;
    if (need > 1.8e19) return fail(HC_EINVAL, "sketch too large");
    uint64_t cells = (uint64_t)need;
    if ((double)cells < need) cells++;
    uint64_t rows = (cells + c - 1) / c;
    if (rows < 3) rows = 3;
    hc_params p;
    memset(&p, 0, sizeof(p));
    p.n = n;
    p.k = 3;
    p.c = c;
    p.rows = rows;
    p.seed = seed;
    p.vtype = (uint32_t)vtype;
    Geo g;
    const hc_status s = to_geo(&p, &g);
    if (s != HC_OK) return s;
    *out = p;
    return HC_OK;
}

hc_status hc_geometry_bloom(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                            uint64_t seed, hc_vtype vtype, hc_params* out, double* eps) {
    g_last_error.clear();
    if (out == nullptr) return fail(HC_EINVAL, "out is NULL");
    if (!(gamma > 0.0) || !isfinite(gamma)) return fail(HC_EINVAL, "gamma must be > 0");
    if (c == 0 || c > 1024 || (c & (c - 1)) != 0)
        return fail(HC_EINVAL, "c must be a power of two in [1, 1024]");
    if (n == 0 || n > 0xffffffffull) return fail(HC_EINVAL, "n must be in [1, 2^32 - 1]");
    if (n_nonzero == 0 || n_nonzero >= n) return fail(HC_EINVAL, "n_nonzero must be in [1, n)");
    // section 3.3: eps = 1 / (ln^2 2 * gamma * C * lambda), lambda n zeros,
    // log2(1 / eps) hashes and (n / ln 2) log2(1 / eps) bits
    const double ln2 = log(2.0);
    const double lambda = (double)(n - n_nonzero) / (double)n_nonzero;
    const double e = 1.0 / (ln2 * ln2 * gamma * 32.0 * lambda);
    double k = floor(log2(1.0 / e) + 0.5);
    if (!(k >= 1.0)) return fail(HC_EINVAL, "too dense for a Bloom filter (log2(1/eps) rounds to 0)");
    if (k > 64.0) k = 64.0;
    const double bits = ceil(k * (double)n_nonzero / ln2);
    const uint64_t brows = ((uint64_t)bits + c - 1) / c;
    // the sketch holds the expected candidates: support and false positives
    const double cand = ceil((double)n_nonzero + ldexp(1.0, -(int)k) * (double)(n - n_nonzero));
    const double need = gamma * cand;
    uint64_t cells = (uint64_t)need;
    if ((double)cells < need) cells++;
    uint64_t rows = (cells + c - 1) / c;
    if (rows < 3) rows = 3;
    hc_params p;
    memset(&p, 0, sizeof(p));
    p.n = n;
    p.k = 3;
    p.c = c;
    p.rows = rows;
    p.seed = seed;
    p.vtype = (uint32_t)vtype;
    p.bloom_k = (uint32_t)k;
    p.bloom_rows = brows;
    Geo g;
    const hc_status s = to_geo(&p, &g);
    if (s != HC_OK) return s;
    *out = p;
    if (eps != nullptr) *eps = e;
    return HC_OK;
}

namespace {

// Blocked geometry for a given number of rows per block (validated inputs).
hc_status blocked_for_rows(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                           uint32_t block_rows, uint64_t seed, hc_vtype vtype, hc_params* out) {
    const uint64_t batches = (n + c - 1) / c;
    // batches per block whose expected share of the support, times gamma,
    // fills block_rows rows; whole bitmap words per block
    const double kk = floor((double)block_rows * (double)n / (gamma * (double)n_nonzero));
    uint64_t K = kk < 1.0 ? 1 : (kk > 1e18 ? (uint64_t)1e18 : (uint64_t)kk);
    if (K > kBlockedMaxBatches) K = kBlockedMaxBatches;
    if (K > batches) K = batches;
    const uint64_t unit = c >= 32 ? 1 : 32 / c;
    K -= K % unit;
    if (K == 0) K = unit;
    // rows of one block: sized for the expected share, at most block_rows
    const double share = ceil((double)n_nonzero * (double)(K * c) / (double)n);
    const double need = gamma * share;
    uint64_t cells = (uint64_t)need;
    if ((double)cells < need) cells++;
    uint64_t rb = (cells + c - 1) / c;
    if (rb < 3) rb = 3;
    if (rb > block_rows) rb = block_rows;
    const uint64_t nblocks = (batches + K - 1) / K;
    hc_params p;
    memset(&p, 0, sizeof(p));
    p.n = n;
    p.k = 3;
    p.c = c;
    p.rows = nblocks * rb;
    p.seed = seed;
    p.vtype = (uint32_t)vtype;
    p.block = (uint32_t)K;
    Geo g;
    hc_status s = to_geo(&p, &g);
    if (s != HC_OK) return s;
    if ((s = blocked_supported(g)) != HC_OK) return s;
    *out = p;
    return HC_OK;
}

}  // namespace

hc_status hc_geometry_blocked(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                              uint32_t block_rows, uint64_t seed, hc_vtype vtype, hc_params* out) {
    g_last_error.clear();
    if (out == nullptr) return fail(HC_EINVAL, "out is NULL");
    if (!(gamma > 0.0) || !isfinite(gamma)) return fail(HC_EINVAL, "gamma must be > 0");
    if (c == 0 || c > 1024 || (c & (c - 1)) != 0)
        return fail(HC_EINVAL, "c must be a power of two in [1, 1024]");
    if (n == 0 || n > 0xffffffffull) return fail(HC_EINVAL, "n must be in [1, 2^32 - 1]");
    if (n_nonzero == 0 || n_nonzero > n) return fail(HC_EINVAL, "n_nonzero must be in [1, n]");
    if (block_rows != 0 && block_rows < 3) return fail(HC_EINVAL, "block_rows must be 0 or >= 3");
    if (block_rows != 0) return blocked_for_rows(n, n_nonzero, gamma, c, block_rows, seed, vtype, out);
    DeviceInfo di;
    const hipError_t e = device_info(&di);
    if (e != hipSuccess) return fail_hip(e, "hc_geometry_blocked");
    // A block peels like a random hypergraph only when its batch-to-row graph
    // is large: with few batches per block and dense batches, the graph's
    // short cycles line up whole columns of elements into stopping sets.
    // Measured at gamma = 1.3 (aggregate density d from 6 % to 73 %), blocks of
    // K >= 600 d batches all peeled; fewer failed for d >= 0.4.  Halve c (not
    // below 32, where a block's batches still get distinct rotation offsets)
    // until the blocks hold that many batches.
    const double density = (double)n_nonzero / (double)n;
    hc_params best;
    memset(&best, 0, sizeof(best));
    for (uint32_t cc = c;; cc /= 2) {
        // each block is one workgroup of the encode and of the decode, whose
        // time grows with its batches K, and the blocks run ceil(nblocks /
        // CUs) workgroups deep per CU: take the row count minimising that
        // product (ties to more rows: fewer, larger blocks peel more
        // reliably), among blocks of 10,240 to 20,480 cells (below about ten
        // thousand members a block needs more room than gamma = 1.3)
        bool found = false;
        uint64_t best_cost = 0;
        hc_params pick;
        memset(&pick, 0, sizeof(pick));
        for (uint32_t br = (10240 + cc - 1) / cc; br <= (20480 + cc - 1) / cc; br++) {
            if (br < 3) continue;
            hc_params p;
            if (blocked_for_rows(n, n_nonzero, gamma, cc, br, seed, vtype, &p) != HC_OK) continue;
            const uint64_t batches = (n + cc - 1) / cc;
            const uint64_t nblocks = (batches + p.block - 1) / p.block;
            const uint64_t cost = (nblocks + di.cus - 1) / di.cus * p.block;
            if (!found || cost <= best_cost) {
                pick = p;
                best_cost = cost;
                found = true;
            }
        }
        if (found) best = pick;
        const bool enough = found && (double)pick.block >= 600.0 * density;
        if (enough || cc <= 32 || cc == 1) break;
    }
    if (best.n == 0) return fail(HC_EUNSUPPORTED, "no block size fits the LDS kernels");
    g_last_error.clear();
    *out = best;
    return HC_OK;
}

hc_status hc_sizes(const hc_params* p, uint64_t max_support, size_t* y_bytes, size_t* b_bytes,
                   size_t* ws_bytes) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (y_bytes) *y_bytes = (size_t)g.cells * 4;
    if (b_bytes) *b_bytes = (size_t)g.bwords * 4;
    if (ws_bytes)
        *ws_bytes = g.block ? blocked_layout(g).total : decode_layout(g, max_support).total;
    return HC_OK;
}

hc_status hc_encode(const hc_params* p, const void* x, void* y, uint32_t* b, hipStream_t stream) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (!x || !y || !b) return fail(HC_EINVAL, "x, y and b must be non-NULL");
    if (!aligned(x, 4) || !aligned(y, 4) || !aligned(b, 4))
        return fail(HC_EINVAL, "x, y and b must be 4-byte aligned");
    if (g.block) {
        const hc_status bs = blocked_supported(g);
        if (bs != HC_OK) return bs;
        const hipError_t e = launch_encode_blocked(g, x, y, b, stream);
        return e == hipSuccess ? HC_OK : fail_hip(e, "hc_encode");
    }
    const hipError_t e = launch_encode_dense(g, x, y, b, stream);
    return e == hipSuccess ? HC_OK : fail_hip(e, "hc_encode");
}

hc_status hc_encode_gather(const hc_params* p, const void* plan, size_t plan_bytes, const void* x,
                           void* y, uint32_t* b, hipStream_t stream) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (g.block) return fail(HC_EUNSUPPORTED, "a blocked sketch is encoded by hc_encode");
    if (g.bloom_k) return fail(HC_EUNSUPPORTED, "the gathered encode writes a bitmap index");
    if (!plan_supported(g)) return fail(HC_EUNSUPPORTED, "plans need c >= 256");
    if (!plan || !aligned(plan, 256)) return fail(HC_EINVAL, "plan must be non-NULL and 256-byte aligned");
    if (plan_bytes < plan_layout(g).total) return fail(HC_EWORKSPACE, "plan smaller than hc_plan_bytes reports");
    if (!x || !y || !b) return fail(HC_EINVAL, "x, y and b must be non-NULL");
    if (!aligned(x, 4) || !aligned(y, 4) || !aligned(b, 4))
        return fail(HC_EINVAL, "x, y and b must be 4-byte aligned");
    const hipError_t e = launch_encode_gather(g, plan, x, y, b, stream);
    return e == hipSuccess ? HC_OK : fail_hip(e, "hc_encode_gather");
}

hc_status hc_encode_staged_bytes(const hc_params* p, size_t* bytes) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (!bytes) return fail(HC_EINVAL, "bytes is NULL");
    if (g.block) return fail(HC_EUNSUPPORTED, "a blocked sketch is encoded by hc_encode");
    if (!plan_supported(g)) return fail(HC_EUNSUPPORTED, "the staged encode needs c >= 256");
    *bytes = stage_layout(g).total;
    return HC_OK;
}

hc_status hc_encode_staged(const hc_params* p, const void* plan, size_t plan_bytes, void* ws,
                           size_t ws_bytes, const void* x, void* y, uint32_t* b,
                           hipStream_t stream) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (g.block) return fail(HC_EUNSUPPORTED, "a blocked sketch is encoded by hc_encode");
    if (!plan_supported(g)) return fail(HC_EUNSUPPORTED, "the staged encode needs c >= 256");
    if (!plan || !aligned(plan, 256)) return fail(HC_EINVAL, "plan must be non-NULL and 256-byte aligned");
    if (plan_bytes < plan_layout(g).total) return fail(HC_EWORKSPACE, "plan smaller than hc_plan_bytes reports");
    if (!ws || !aligned(ws, 256)) return fail(HC_EINVAL, "ws must be non-NULL and 256-byte aligned");
    if (ws_bytes < stage_layout(g).total)
        return fail(HC_EWORKSPACE, "ws smaller than hc_encode_staged_bytes reports");
    if (!x || !y || !b) return fail(HC_EINVAL, "x, y and b must be non-NULL");
    if (!aligned(x, 4) || !aligned(y, 4) || !aligned(b, 4))
        return fail(HC_EINVAL, "x, y and b must be 4-byte aligned");
    const hipError_t e = launch_encode_staged(g, plan, ws, x, y, b, stream);
    return e == hipSuccess ? HC_OK : fail_hip(e, "hc_encode_staged");
}

hc_status hc_encode_coo(const hc_params* p, const uint32_t* idx, const void* val, uint64_t nnz,
                        void* y, uint32_t* b, hipStream_t stream) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (!y || !b) return fail(HC_EINVAL, "y and b must be non-NULL");
    if (nnz > 0 && (!idx || !val)) return fail(HC_EINVAL, "idx and val must be non-NULL");
    if (!aligned(y, 4) || !aligned(b, 4) || (nnz > 0 && (!aligned(idx, 4) || !aligned(val, 4))))
        return fail(HC_EINVAL, "buffers must be 4-byte aligned");
    const hipError_t e = launch_encode_coo(g, idx, val, nnz, y, b, stream);
    return e == hipSuccess ? HC_OK : fail_hip(e, "hc_encode_coo");
}

hc_status hc_aggregate(const hc_params* p, const void* y_in, const uint32_t* b_in, uint32_t W,
                       void* y_out, uint32_t* b_out, hipStream_t stream) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (W == 0) return fail(HC_EINVAL, "W must be >= 1");
    if (!y_in || !b_in || !y_out || !b_out) return fail(HC_EINVAL, "buffers must be non-NULL");
    if (!aligned(y_in, 4) || !aligned(b_in, 4) || !aligned(y_out, 4) || !aligned(b_out, 4))
        return fail(HC_EINVAL, "buffers must be 4-byte aligned");
    const hipError_t e = launch_aggregate(g, y_in, b_in, W, y_out, b_out, stream);
    return e == hipSuccess ? HC_OK : fail_hip(e, "hc_aggregate");
}

hc_status hc_plan_bytes(const hc_params* p, size_t* bytes) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (!bytes) return fail(HC_EINVAL, "bytes is NULL");
    if (g.block) return fail(HC_EUNSUPPORTED, "a blocked sketch is decoded without a plan");
    if (!plan_supported(g)) return fail(HC_EUNSUPPORTED, "plans need c >= 256");
    *bytes = plan_layout(g).total;
    return HC_OK;
}

hc_status hc_plan_build(const hc_params* p, void* plan, size_t plan_bytes, hipStream_t stream) {
    g_last_error.clear();
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (g.block) return fail(HC_EUNSUPPORTED, "a blocked sketch is decoded without a plan");
    if (!plan_supported(g)) return fail(HC_EUNSUPPORTED, "plans need c >= 256");
    if (!plan || !aligned(plan, 256)) return fail(HC_EINVAL, "plan must be non-NULL and 256-byte aligned");
    if (plan_bytes < plan_layout(g).total) return fail(HC_EWORKSPACE, "plan smaller than hc_plan_bytes reports");
    const hipError_t e = launch_plan_build(g, plan, stream);
    return e == hipSuccess ? HC_OK : fail_hip(e, "hc_plan_build");
}

}  // extern "C"

namespace {

// hc_decode's argument checks, workspace check and launches.  ws == nullptr
// means the static scratch array below (hc_decode_noalloc).
hc_status decode_impl(const hc_params* p, const void* plan, const void* y_agg,
                      const uint32_t* b_agg, void* x_out, uint32_t* coo_idx, void* coo_val,
                      uint64_t coo_cap, uint32_t* mask, hc_decode_info* info,
                      uint64_t max_support, void* ws, size_t ws_bytes, hipStream_t stream);

}  // namespace

extern "C" {

hc_status hc_decode(const hc_params* p, const void* plan, const void* y_agg,
                    const uint32_t* b_agg, void* x_out, uint32_t* coo_idx, void* coo_val,
                    uint64_t coo_cap, uint32_t* mask, hc_decode_info* info, uint64_t max_support,
                    void* ws, size_t ws_bytes, hipStream_t stream) {
    g_last_error.clear();
    if (!ws) return fail(HC_EINVAL, "ws must be non-NULL");
    return decode_impl(p, plan, y_agg, b_agg, x_out, coo_idx, coo_val, coo_cap, mask, info,
                       max_support, ws, ws_bytes, stream);
}

hc_status hc_decode_noalloc(const hc_params* p, const void* plan, const void* y_agg,
                            const uint32_t* b_agg, void* x_out, uint32_t* coo_idx,
                            void* coo_val, uint64_t coo_cap, uint32_t* mask,
                            hc_decode_info* info, uint64_t max_support, hipStream_t stream) {
    g_last_error.clear();
    return decode_impl(p, plan, y_agg, b_agg, x_out, coo_idx, coo_val, coo_cap, mask, info,
                       max_support, nullptr, 0, stream);
}

}  // extern "C"

namespace {

// The allocation-free decode's workspace: one array per GPU, held by the
// loaded library until the process ends.  Host code never passes its name to
// a kernel (in host code it is only a stand-in for the device symbol): the
// device address comes from hipGetSymbolAddress, once per device, and the
// kernels take that.  Every hc_decode_noalloc call on a GPU shares the array;
// the decode clears what it needs cleared itself.
__device__ __align__(256) unsigned char scratch[HC_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_ptr;  // device -> address of its copy of `scratch`

hc_status scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail_hip(e, "hc_decode_noalloc: hipGetDevice");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch_ptr.find(dev);
    if (it == g_scratch_ptr.end()) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return fail_hip(e, "hc_decode_noalloc: hipGetSymbolAddress");
        if (ptr == nullptr || !aligned(ptr, 256))
            return fail(HC_EHIP, "hc_decode_noalloc: scratch has no usable device address");
        it = g_scratch_ptr.emplace(dev, ptr).first;
    }
    *out = it->second;
    return HC_OK;
}

hc_status decode_impl(const hc_params* p, const void* plan, const void* y_agg,
                      const uint32_t* b_agg, void* x_out, uint32_t* coo_idx, void* coo_val,
                      uint64_t coo_cap, uint32_t* mask, hc_decode_info* info,
                      uint64_t max_support, void* ws, size_t ws_bytes, hipStream_t stream) {
    Geo g;
    const hc_status s = to_geo(p, &g);
    if (s != HC_OK) return s;
    if (plan && g.block) return fail(HC_EINVAL, "a blocked sketch is decoded without a plan");
    if (plan && (!plan_supported(g) || !aligned(plan, 256)))
        return fail(HC_EINVAL, "plan given for a geometry with c < 256, or not 256-byte aligned");
    if (!y_agg || !b_agg || !info) return fail(HC_EINVAL, "y_agg, b_agg and info must be non-NULL");
    if (!aligned(y_agg, 4) || !aligned(b_agg, 4) || (x_out && !aligned(x_out, 4)) ||
        (mask && !aligned(mask, 4)) || (coo_idx && !aligned(coo_idx, 4)) ||
        (coo_val && !aligned(coo_val, 4)))
        return fail(HC_EINVAL, "buffers must be 4-byte aligned");
    if ((ws && !aligned(ws, 256)) || !aligned(info, 8))
        return fail(HC_EINVAL, "ws must be 256-byte and info 8-byte aligned");
    if ((coo_idx == nullptr) != (coo_val == nullptr))
        return fail(HC_EINVAL, "coo_idx and coo_val must both be given or both be NULL");
    DecodeOut out;
    out.x_out = x_out;
    out.coo_idx = coo_idx;
    out.coo_val = coo_val;
    out.coo_cap = coo_cap;
    out.mask = mask;
    out.info = info;
    const char* where = ws ? "hc_decode" : "hc_decode_noalloc";
    const size_t need = g.block ? blocked_layout(g).total : decode_layout(g, max_support).total;
    if (ws == nullptr) {
        // the static scratch array stands in for the caller's workspace
        if (need > (size_t)HC_NOALLOC_SCRATCH_BYTES) {
            char msg[160];
            snprintf(msg, sizeof(msg),
                     "hc_decode_noalloc: this decode needs %zu bytes of workspace, more than the "
                     "%zu of its static scratch (use hc_decode)",
                     need, (size_t)HC_NOALLOC_SCRATCH_BYTES);
            return fail(HC_EWORKSPACE, msg);
        }
        const hc_status ss = scratch_address(&ws);
        if (ss != HC_OK) return ss;
        ws_bytes = HC_NOALLOC_SCRATCH_BYTES;
    }
    if (g.block) {
        const hc_status bs = blocked_supported(g);
        if (bs != HC_OK) return bs;
        const BlockedLayout BL = blocked_layout(g);
        if (ws_bytes < BL.total) return fail(HC_EWORKSPACE, "workspace smaller than hc_sizes reports");
        const hipError_t e = launch_decode_blocked(g, y_agg, b_agg, out, BL, ws, stream);
        return e == hipSuccess ? HC_OK : fail_hip(e, where);
    }
    const DecodeLayout L = decode_layout(g, max_support);
    if (ws_bytes < need) return fail(HC_EWORKSPACE, "workspace smaller than hc_sizes reports");
    const hipError_t e = launch_decode(g, plan, y_agg, b_agg, out, L, ws, stream);
    return e == hipSuccess ? HC_OK : fail_hip(e, where);
}

}  // namespace
