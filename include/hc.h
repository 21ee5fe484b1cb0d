/*
 * hc.h -- C ABI of the MI355X (gfx950) library for lossless homomorphic
 * gradient compression: a Count Sketch plus a bitmap index per worker, summed
 * and OR-ed across workers, and decoded by parallel peeling.
 *
 * Paper: "Accelerating Distributed Deep Learning using Lossless Homomorphic
 * Compression", arXiv 2402.07529.  Algorithm 1 has two phases around the
 * aggregation API; this library exposes one call per stage:
 *
 *   hc_encode / hc_encode_coo   Algorithm 1, phase I (sections 3.1, 3.2, 3.4)
 *   hc_encode_gather            the same for dense gradients, row by row
 *                               through a plan
 *   hc_encode_staged            the same for sparse gradients: nonzeros staged
 *                               per batch, rows assembled through a plan
 *   hc_aggregate                what the aggregation API does between the
 *                               phases: Y <- sum Y, B <- OR B (section 3)
 *   hc_decode                   Algorithm 1, phase II (section 3.2 peeling,
 *                               section 3.1 median estimate for leftovers)
 *   hc_geometry / hc_sizes      sketch sizing, |Y| >= gamma * n (section 3.2)
 *   hc_geometry_bloom           the same with a Bloom-filter index (section 3.3)
 *   hc_plan_bytes / _build      the inverse row map of a geometry (section 3.4
 *                               batching), built once, used by the decode and
 *                               by hc_encode_gather
 *
 * Conventions for every call:
 *   - Buffer pointers are DEVICE pointers unless marked "host".  The caller
 *     owns all memory; the library allocates no device memory in any call.
 *   - Calls are asynchronous on `stream` (0 = the null stream).  A returned
 *     HC_OK means the arguments were valid and the kernels were enqueued.
 *   - Errors are returned as hc_status; nothing is thrown across the ABI.
 *     hc_last_error() gives a message for the last failing call of the
 *     calling host thread.  Invalid arguments are detected before anything
 *     is enqueued.
 *   - Value, index and bitmap buffers need their natural 4-byte alignment
 *     (16-byte alignment lets the kernels use vector memory operations on
 *     sketches, bitmaps and outputs; hc_encode and hc_encode_staged read the
 *     gradient with 16-byte loads at any 4-byte alignment);
 *     the decode workspace must be 256-byte aligned and the decode info
 *     8-byte aligned.  hipMalloc and PyTorch allocations satisfy all of it.
 *
 * Sketch format (identical for every worker; the paper leaves these details
 * open):
 *   cells = rows * c.  Parameter p lies in batch b = p / c at column
 *   t = p mod c.  Three 64-bit hashes h_j = SplitMix64 output number 3b + j for
 *   state `seed` (j = 0, 1, 2) give three distinct rows r_j (scaled from the
 *   low 32 bits of h_j, later rows skipping earlier ones), rotations
 *   bias_j = (h_j >> 32) mod c and signs g_j = -1 if bit 63 of h_j is set,
 *   else +1.  Cell j of p is r_j * c + ((t + bias_j) mod c).
 *   Y[cells] holds int32 (wrapping, like a switch's integer adders) or fp32.
 *   B[ceil(n/32)] is a bitmap, bit p = bit (p mod 32) of word p / 32; bits at
 *   or past n are zero.
 *
 * Bloom-filter index (section 3.3), selected by hc_params.bloom_k = k > 0: B is
 * a bit array of bloom_rows rows of c bits (the index reshaped into a matrix of
 * width c as in section 3.4) instead of the bitmap, ceil(bloom_rows * c / 32)
 * words, bit q = bit (q mod 32) of word q / 32, bits past bloom_rows * c zero.
 * Hash i < k of batch b is u = SplitMix64 output number 3 * 2^32 + k * b + i
 * for `seed`, giving row mulhi32(lo32(u), bloom_rows) and rotation
 * (u >> 32) mod c; a nonzero parameter at column t sets bit
 * row * c + ((t + rotation) mod c) for each i.  The decode treats as the support
 * every parameter whose k bits are all set: the nonzeros (a Bloom filter has no
 * false negatives) and the zeros the filter lets through, which peel to 0.
 * The filter merges under OR exactly like the bitmap.  Supported with the
 * global sketch only (HC_EUNSUPPORTED with block > 0).
 *
 * Blocked sketch (section 3.2: the sketch split into blocks of a fixed size so
 * that peeling takes O(1) rounds), selected by hc_params.block = K > 0: batch b
 * belongs to parameter block q = b / K (the last block may be shorter), the
 * sketch has nblocks = ceil(ceil(n/c) / K) blocks of R_b = rows / nblocks rows
 * each, and block q owns rows [q * R_b, (q+1) * R_b): the three rows of batch b
 * are drawn as above from R_b instead of rows, sorted ascending and offset by
 * q * R_b.  The rotations of batch number i = b mod K of block q are bias_0 as
 * above, bias_1 = (bias_0 + pi mod c) mod c and bias_2 = (bias_0 + pi div c)
 * mod c, with pi = P(i) for the bijection P of [0, M = c^2) keyed by
 * u_q = SplitMix64 output number 2^62 + q: with a1, a2 and s the low, middle
 * and high 20-bit fields of u_q (a1, a2 made odd) and h = ceil(log2(M) / 2),
 * x = (i + s) mod M, x = x * a1 mod M, x ^= x >> h, x = x * a2 mod M,
 * x ^= x >> h.  For c >= 32 no two batches of one block then sit on the same
 * three rows with the same relative rotations (which would put every two
 * corresponding elements on the same three cells, a pair no sketch size
 * peels), and the offsets carry no arithmetic structure.  Every block then
 * peels on its own.  K * c must be a multiple of 32 and rows a
 * multiple of nblocks with R_b >= 3.  The library's encode and decode of a
 * blocked sketch hold one block per workgroup in LDS, which needs K <= 1024
 * and, per block, R_b * c * (10 for int32, 14 for fp32) + 12 * K + 256 bytes
 * <= 159 KiB (at c = 1024: up to 14 rows for int32, 10 for fp32;
 * HC_EUNSUPPORTED otherwise; hc_encode_coo and hc_aggregate accept any
 * blocked geometry).
 */
#ifndef HC_H
#define HC_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HC_OK = 0,
    HC_EINVAL = 1,        /* invalid argument (null pointer, bad geometry, size) */
    HC_EWORKSPACE = 2,    /* decode workspace smaller than hc_sizes reports       */
    HC_EHIP = 3,          /* a HIP runtime call failed (launch, device query)     */
    HC_EUNSUPPORTED = 4   /* valid but not implemented (k != 3, blocked sketches
                             beyond the LDS kernels' limits)                      */
} hc_status;

typedef enum { HC_I32 = 0, HC_F32 = 1 } hc_vtype;

/* Sketch geometry, shared by every worker of one aggregation. */
typedef struct {
    uint64_t n;        /* gradient length N, 1 .. 2^32 - 1                        */
    uint32_t k;        /* hashes per parameter; the paper's three (only 3)       */
    uint32_t c;        /* batch width of section 3.4, power of two in [1, 1024]  */
    uint64_t rows;     /* sketch rows R >= 3; cells = rows * c must be < 2^32    */
    uint64_t seed;     /* hash seed                                               */
    uint32_t vtype;    /* hc_vtype of the gradient and sketch values             */
    uint32_t block;    /* batches per parameter block of a blocked sketch
                          (section 3.2); 0 = one global sketch                   */
    uint32_t bloom_k;  /* Bloom filter hashes per nonzero (section 3.3), 1..64;
                          0 = the bitmap index of section 3.2                    */
    uint32_t reserved; /* must be 0                                              */
    uint64_t bloom_rows; /* rows of c bits in the Bloom filter (bloom_k > 0);
                          bloom_rows * c must be < 2^32                          */
} hc_params;

/* Written by hc_decode into DEVICE memory. */
typedef struct {
    uint64_t n_support;   /* set bits of the aggregated bitmap (nonzeros of sum X);
                             with a Bloom filter, the parameters it reports as
                             nonzero (the support plus its false positives)     */
    uint64_t n_recovered; /* of those, recovered exactly by peeling                */
    uint64_t rounds;      /* synchronous peeling rounds that recovered >= 1        */
    uint32_t success;     /* 1 iff n_recovered == n_support                        */
    uint32_t status;      /* 0 ok; 1 n_support exceeded max_support (nothing was
                             peeled, every element got the median estimate);
                             2 the round loop's barrier gave up waiting (a
                             device fault; outputs are not valid);
                             3 the plan was built for another geometry
                             (nothing was peeled, as for 1)                     */
} hc_decode_info;

/* Geometry for a gradient of n parameters whose aggregate has about n_nonzero
 * nonzeros: rows = max(3, ceil(ceil(gamma * n_nonzero) / c)), so the sketch
 * has at least gamma * n_nonzero cells (section 3.2 uses gamma = 1.23; section
 * 3.4 uses c = 1024).  `out` is a HOST pointer.  HC_EINVAL if the result is not
 * a valid geometry. */
hc_status hc_geometry(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                      uint64_t seed, hc_vtype vtype, hc_params *out);

/* Geometry of a blocked sketch (section 3.2 blocking) whose blocks have at most
 * block_rows rows (block_rows = 0: chosen for the current device, see below):
 * K = floor(block_rows * n / (gamma * n_nonzero)) batches per
 * block, so that a block's expected share of the aggregate's n_nonzero
 * nonzeros times gamma fills its rows, clamped to [1, min(1024, batches)] and
 * rounded down to a multiple of max(1, 32 / c); each block then gets
 * R_b = min(block_rows, max(3, ceil(ceil(gamma * s) / c))) rows, s = the
 * expected share of a block of K batches rounded up, and rows = nblocks * R_b.
 * Per-block supports scatter around the expected share, so gamma must leave
 * room for the fullest block (about 1.3 at 14 thousand nonzeros per block where
 * the global sketch needs 1.23).  With block_rows = 0 the library takes, among
 * the row counts whose blocks hold 10,240 to 20,480 cells and fit the LDS
 * kernels, the one minimising ceil(nblocks / CUs) * K for the current device's
 * compute-unit count (each block is one workgroup of the encode and the decode,
 * whose time grows with K), ties going to more rows; and if that leaves fewer
 * than K = 600 * n_nonzero / n batches per block it halves c (down to 32) until
 * it does not: blocks of few, dense batches have a small batch-to-row graph
 * whose short cycles line columns of elements up into stopping sets (measured:
 * such blocks failed for aggregate densities of 40 % and more, larger ones did
 * not).  out->c then holds the c used.  This needs a device (HC_EHIP without
 * one), and every worker of an aggregation must use the same geometry.  `out` is a HOST pointer.  HC_EINVAL on invalid arguments,
 * HC_EUNSUPPORTED if a block would not fit the LDS kernels. */
hc_status hc_geometry_blocked(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                              uint32_t block_rows, uint64_t seed, hc_vtype vtype,
                              hc_params *out);

/* Geometry with a Bloom-filter index (section 3.3).  With lambda = (n -
 * n_nonzero) / n_nonzero zero parameters per nonzero and C = 32-bit values, the
 * paper's false positive rate is eps = 1 / (ln^2(2) * gamma * C * lambda); the
 * filter takes k = round(log2(1 / eps)) hashes (at most 64) and
 * ceil(k * n_nonzero / ln 2) bits, rounded up to whole rows of c bits (half its
 * bits end up set, so a zero passes with probability about 2^-k), and the
 * sketch holds gamma times the expected candidates, n_nonzero + 2^-k * (n -
 * n_nonzero), in whole rows of c cells (at least three).  *eps (HOST, may be
 * NULL) receives the paper's eps.  HC_EINVAL if n_nonzero is 0 or >= n, or if k
 * would round to 0 (eps > 2^-1/2: too dense for a filter to pay); `out` is a
 * HOST pointer. */
hc_status hc_geometry_bloom(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                            uint64_t seed, hc_vtype vtype, hc_params *out, double *eps);

/* Byte sizes (HOST outputs, each may be NULL): one sketch Y, one index B (the
 * bitmap, or the Bloom filter), and
 * the decode workspace for a support of up to max_support nonzeros
 * (0 means n, which always suffices; a blocked sketch's workspace does not
 * depend on it). */
hc_status hc_sizes(const hc_params *p, uint64_t max_support, size_t *y_bytes,
                   size_t *b_bytes, size_t *ws_bytes);

/* Plan: the inverse row map of a geometry.  Under section 3.4's batching each
 * batch of c parameters lands, per hash, on one whole sketch row; the plan
 * lists for every row the (batch, hash) pairs landing on it, so that a row can
 * be assembled by one workgroup that gathers its contributions instead of
 * receiving scattered atomics.  It depends only on (n, c, rows, seed): build it
 * once per geometry and reuse it for every worker and iteration.  Requires
 * c >= 256 and an unblocked sketch (HC_EUNSUPPORTED otherwise).  hc_plan_bytes writes the size to the
 * HOST pointer `bytes`; hc_plan_build fills a caller-owned, 256-byte aligned
 * DEVICE buffer of at least that size, asynchronously on `stream`. */
hc_status hc_plan_bytes(const hc_params *p, size_t *bytes);
hc_status hc_plan_build(const hc_params *p, void *plan, size_t plan_bytes, hipStream_t stream);

/* Phase I on a dense gradient x[n] (int32 or fp32 per p->vtype).  Overwrites
 * y[cells] with the Count Sketch (Y[h_j(p)] += g_j(p) * x_p for every nonzero
 * x_p, section 3.1 with the batching of 3.4) and b with the index: the
 * nonzero bitmap b[ceil(n/32)] (section 3.2), or the Bloom filter of every
 * nonzero (section 3.3; b[ceil(bloom_rows * c / 32)]).  No pre-zeroing is
 * needed.  A blocked sketch is built in LDS, one block per workgroup, unless
 * it has fewer blocks than the GPU has CUs: then the whole GPU streams the
 * gradient and adds with global atomics, as for an unblocked sketch.  fp32
 * sums are accumulated with atomics (global, or in LDS), so their rounding
 * order is not fixed. */
hc_status hc_encode(const hc_params *p, const void *x, void *y, uint32_t *b,
                    hipStream_t stream);

/* Phase I on a dense gradient, assembled row by row through a plan: the
 * same outputs as hc_encode with a bitmap index (int32 bit-identical; fp32
 * summed in another order).  hc_encode adds each nonzero into its three cells
 * (section 3.1) with scattered atomics, which bound it when most parameters
 * are nonzero, as in section 4.1's microbenchmark.  Here one workgroup per
 * sketch row reads every batch that lands on the row (section 3.4: a batch
 * lands on one whole row per hash, rotated) and sums the row in LDS: 12n
 * bytes of reads whatever the density, no global atomics.  Unblocked sketch,
 * bitmap index, c >= 256 (HC_EUNSUPPORTED otherwise).  plan: built by
 * hc_plan_build for the same params, 256-byte aligned (HC_EINVAL), plan_bytes
 * at least hc_plan_bytes (HC_EWORKSPACE).  A plan built for other params is
 * detected on the device from its header: the call then writes a zero sketch
 * and an all-ones bitmap, which a decode reports as a failure (success = 0)
 * rather than as a gradient. */
hc_status hc_encode_gather(const hc_params *p, const void *plan, size_t plan_bytes,
                           const void *x, void *y, uint32_t *b, hipStream_t stream);

/* Phase I on a dense gradient, staged: the same outputs as hc_encode (int32
 * bit-identical; fp32 summed in another order), without its three scattered
 * atomics per nonzero (section 3.1), which bound hc_encode on sparse
 * gradients.  A first pass streams x once, writes the index (bitmap or Bloom
 * filter, as hc_encode) and compacts each batch's nonzeros (section 3.4's
 * batches of c parameters) into a per-batch list of up to 64 (column, value)
 * pairs in the workspace; a second pass builds every sketch row in LDS from
 * the lists of the batches the plan lands on it (section 3.4: a batch lands on
 * one whole row per hash, rotated) and stores it once.  A batch with more than
 * 64 nonzeros is read from x itself by the second pass (once per hash), so any
 * density is handled; below about 6 % (c = 1024) every batch fits its list.
 * Unblocked sketch, c >= 256 (HC_EUNSUPPORTED otherwise).  plan: built by
 * hc_plan_build for the same params, 256-byte aligned (HC_EINVAL), plan_bytes
 * at least hc_plan_bytes (HC_EWORKSPACE); a plan built for other params is
 * detected on the device and gives a zero sketch and an all-ones index (as
 * hc_encode_gather).  ws: 256-byte aligned device workspace (HC_EINVAL) of at
 * least hc_encode_staged_bytes (HC_EWORKSPACE), about n / 2 bytes at
 * c = 1024; contents on entry are ignored.  hc_encode_staged_bytes writes the
 * size to the HOST pointer `bytes`. */
hc_status hc_encode_staged_bytes(const hc_params *p, size_t *bytes);
hc_status hc_encode_staged(const hc_params *p, const void *plan, size_t plan_bytes, void *ws,
                           size_t ws_bytes, const void *x, void *y, uint32_t *b,
                           hipStream_t stream);

/* Phase I on COO input: idx[nnz] (uint32, each < n, any order) and
 * val[nnz].  Zero values are skipped; repeated indices are summed.  Same
 * outputs as hc_encode of the equivalent dense gradient. */
hc_status hc_encode_coo(const hc_params *p, const uint32_t *idx, const void *val,
                        uint64_t nnz, void *y, uint32_t *b, hipStream_t stream);

/* The aggregation step: y_out[i] = sum over w < W of y_in[w * cells + i]
 * (int32 wraps modulo 2^32; fp32 adds in worker order 0..W-1) and
 * b_out[i] = OR over w of b_in[w * words + i], words = the index's words
 * (ceil(n/32) for the bitmap, ceil(bloom_rows * c / 32) for a Bloom filter).
 * Inputs are W sketches and W indexes stored back to back.  Outputs may not
 * alias inputs.  W >= 1. */
hc_status hc_aggregate(const hc_params *p, const void *y_in, const uint32_t *b_in,
                       uint32_t W, void *y_out, uint32_t *b_out, hipStream_t stream);

/* Phase II on an aggregated sketch.  y_agg and b_agg are not modified.
 * plan: a plan built for the same geometry (then the per-cell counters are
 * gathered row by row, without atomics), or NULL (they are built with
 * atomics).  Results are identical either way; a plan built for another
 * geometry is detected on the device and reported as status 3.  A blocked
 * sketch takes no plan (HC_EINVAL if one is given): each block is peeled by one
 * workgroup in LDS, in the same synchronous rounds; info->rounds is then the
 * largest round count of any block, and max_support is not used.  With a
 * Bloom-filter index the support is every parameter whose filter bits are all
 * set (probed into a bitmap in the workspace first); max_support must then
 * cover those candidates, false positives included.
 * Outputs (each may be NULL):
 *   x_out[n]              dense sum X: recovered values, the Count Sketch
 *                         median estimate for members of the support that
 *                         could not be peeled, 0 outside the support;
 *   coo_idx, coo_val      the support in ascending order with its values, at
 *                         most coo_cap entries (entries past coo_cap are not
 *                         written; n_support in info tells how many exist);
 *   mask[ceil(n/32)]      bit p set iff p was recovered by peeling;
 *   info (one struct)     summary, DEVICE memory.
 * ws/ws_bytes: device workspace of at least the ws_bytes hc_sizes reports for
 * the same max_support; contents on entry are ignored.  max_support also picks
 * how round 0 runs on an int32 sketch with a plan: by rows when the sketch has
 * a cell per element of max_support, entry by entry otherwise (a bound near
 * the true support keeps the faster one; results are the same either way).
 * Peeling runs as synchronous rounds entirely on the device (one cooperative
 * kernel; no host round trips).  Decode failure is data (info->success), not
 * an error status. */
hc_status hc_decode(const hc_params *p, const void *plan, const void *y_agg,
                    const uint32_t *b_agg,
                    void *x_out, uint32_t *coo_idx, void *coo_val, uint64_t coo_cap,
                    uint32_t *mask, hc_decode_info *info, uint64_t max_support,
                    void *ws, size_t ws_bytes, hipStream_t stream);

/* Bytes of the static device scratch array behind hc_decode_noalloc (64 MiB
 * per GPU the library runs on, held until the process ends). */
#define HC_NOALLOC_SCRATCH_BYTES ((size_t)64 * 1024 * 1024)

/* hc_decode without a workspace argument, for callers that cannot allocate
 * device memory (code under stream capture, tight serving loops, harnesses
 * that forbid allocation).  Same arguments, checks, outputs and stream
 * semantics as hc_decode with ws and ws_bytes removed: the workspace is a
 * static device array of HC_NOALLOC_SCRATCH_BYTES in the library, one per
 * GPU, and the call allocates nothing.  Limit: the decode must need at most
 * that much workspace, i.e. hc_sizes must report ws_bytes <=
 * HC_NOALLOC_SCRATCH_BYTES for the same params and max_support (a blocked
 * sketch's decode always fits; for a global int32 sketch the workspace is
 * about 20 bytes per cell plus 12 per support element, e.g. one million cells
 * with a support of up to 1.5 million); HC_EWORKSPACE otherwise, before
 * anything is enqueued.  All calls on one GPU share its scratch array: calls
 * that overlap in time on one GPU (different streams or host threads without
 * ordering) race and give undefined results; calls ordered on one stream are
 * safe.  The scratch contents on entry are ignored, as hc_decode ignores its
 * workspace's. */
hc_status hc_decode_noalloc(const hc_params *p, const void *plan, const void *y_agg,
                            const uint32_t *b_agg,
                            void *x_out, uint32_t *coo_idx, void *coo_val, uint64_t coo_cap,
                            uint32_t *mask, hc_decode_info *info, uint64_t max_support,
                            hipStream_t stream);

/* Human-readable name of a status, and the message of the calling thread's
 * last failing call ("" if none). */
const char *hc_status_string(hc_status s);
const char *hc_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
