// hc_internal.h -- host-side launchers of the gfx950 kernels (internal to
// libhc; the public surface is include/hc.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hc {

// Validated geometry in the form the kernels take it.
struct Geo {
    uint64_t n;       // gradient length
    uint64_t words;   // ceil(n / 32)
    uint32_t rows;    // R
    uint32_t c;       // batch width (power of two)
    uint32_t cmask;   // c - 1
    uint32_t log2c;
    uint32_t cells;   // rows * c
    uint64_t seed;
    bool f32;         // value type: fp32 (else int32)
    // blocked sketch (section 3.2): block batches per parameter block, each
    // block owning brows consecutive rows; block == 0 is one global sketch
    // (then brows == rows and nblocks == 1)
    uint32_t block;
    uint32_t brows;
    uint32_t nblocks;
    // index: the bitmap (bloom_k == 0) or a Bloom filter of bloom_rows rows of
    // c bits (section 3.3); bwords = words of the index
    uint32_t bloom_k;
    uint32_t bloom_rows;
    uint64_t bwords;
};

struct DeviceInfo {
    int cus;          // compute units
};
// Properties of the current device, queried once per device (thread-safe).
hipError_t device_info(DeviceInfo* out);
// Resident workgroups per CU of `kernel` at `block` lanes and no dynamic LDS
// on the current device (at least 1), queried once per (device, kernel,
// block) and cached (thread-safe).
hipError_t occupancy_per_cu(const void* kernel, int block, int* out);
// Lets `kernel` take up to `bytes` of dynamic LDS on the current device (set
// once per (device, kernel), thread-safe).
hipError_t allow_dynamic_lds(const void* kernel, int bytes);

// Bloom filter: candidate bitmap cand[words] of the parameters whose bloom_k
// filter bits are all set
hipError_t launch_bloom_probe(const Geo& g, const uint32_t* filter, uint32_t* cand,
                              hipStream_t s);

// encode
hipError_t launch_fill_u32(uint32_t* p, uint64_t count, uint32_t value, hipStream_t s);
hipError_t launch_encode_dense(const Geo& g, const void* x, void* y, uint32_t* b,
                               hipStream_t s);
hipError_t launch_encode_coo(const Geo& g, const uint32_t* idx, const void* val,
                             uint64_t nnz, void* y, uint32_t* b, hipStream_t s);
// dense encode gathered row by row through a plan (c >= 256, bitmap index,
// unblocked sketch)
hipError_t launch_encode_gather(const Geo& g, const void* plan, const void* x, void* y,
                                uint32_t* b, hipStream_t s);

// staged dense encode (c >= 256, unblocked sketch): a first pass writes the
// index and, per batch of c parameters, its nonzero count and up to kStageCap
// of its (column, value) pairs into a caller workspace; a second pass builds
// every sketch row in LDS through the plan
constexpr uint32_t kStageCap = 64;
struct StageLayout {
    uint64_t nb;          // batches
    size_t count, list, total;
};
StageLayout stage_layout(const Geo& g);
hipError_t launch_encode_staged(const Geo& g, const void* plan, void* ws, const void* x, void* y,
                                uint32_t* b, hipStream_t s);
hipError_t launch_fill2_u32(uint32_t* p, uint64_t count, uint32_t* p2, uint64_t count2,
                            uint32_t value, hipStream_t s);

// aggregate
hipError_t launch_aggregate(const Geo& g, const void* y_in, const uint32_t* b_in, uint32_t W,
                            void* y_out, uint32_t* b_out, hipStream_t s);

// inverse row map of a geometry ("plan"), built once per geometry
constexpr uint32_t kPlanMagic = 0x31706368u;  // "hcp1"
struct PlanHeader {
    uint64_t n;
    uint64_t seed;
    uint32_t c;
    uint32_t rows;
    uint32_t magic;
    uint32_t pad;
};
struct PlanLayout {
    uint64_t nb;       // batches
    uint64_t ntiles;   // scan tiles over the rows
    size_t header, rowoff, entry, rowcnt, tiles, total;
};
PlanLayout plan_layout(const Geo& g);
bool plan_supported(const Geo& g);  // c >= 256
hipError_t launch_plan_build(const Geo& g, void* plan, hipStream_t s);

// blocked sketch, one workgroup per block with the block's sketch in LDS
constexpr uint32_t kBlockedMaxBatches = 1024;  // packed LDS counters: deg * 2^20 + sum of batches
constexpr size_t kLdsBytes = 163840;           // LDS per workgroup on gfx950
constexpr size_t kLdsReserve = 1024;           // for the kernels' own static LDS
size_t blocked_encode_lds(const Geo& g);
size_t blocked_decode_lds(const Geo& g);
struct BlockedLayout {
    uint64_t nchunks;
    size_t ctrl, bctrl, blk, total;
};
BlockedLayout blocked_layout(const Geo& g);
hipError_t launch_encode_blocked(const Geo& g, const void* x, void* y, uint32_t* b,
                                 hipStream_t s);

// decode workspace layout (byte offsets into the caller's workspace)
struct DecodeLayout {
    uint64_t cap;       // max support the workspace holds
    uint64_t nchunks;   // bitmap chunks of kChunkWords words
    uint64_t ntiles;    // tiles of the support passes (a few chunks each)
    size_t ctrl, sync, blk, cpre, tcnt, woffb, elem, vals, peeled, cnt, yw, queue, mark, cand, total;
};
constexpr uint32_t kChunkWords = 1024;
DecodeLayout decode_layout(const Geo& g, uint64_t max_support);

struct DecodeOut {
    void* x_out;
    uint32_t* coo_idx;
    void* coo_val;
    uint64_t coo_cap;
    uint32_t* mask;
    void* info;   // hc_decode_info*
};
// plan: an inverse row map built for g, or nullptr (then the per-cell
// counters are built with atomics)
hipError_t launch_decode(const Geo& g, const void* plan, const void* y_agg,
                         const uint32_t* b_agg, const DecodeOut& out, const DecodeLayout& L,
                         void* ws, hipStream_t s);
hipError_t launch_decode_blocked(const Geo& g, const void* y_agg, const uint32_t* b_agg,
                                 const DecodeOut& out, const BlockedLayout& L, void* ws,
                                 hipStream_t s);
// support offsets of the bitmap chunks: blk[i] = set bits before chunk i of
// kChunkWords words; ctrl is a 64-byte control block that the scan also uses
hipError_t launch_support_offsets(const Geo& g, const uint32_t* b, uint32_t* blk, void* ctrl,
                                  hipStream_t s);

}  // namespace hc
