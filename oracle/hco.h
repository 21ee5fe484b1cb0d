/*
 * hco.h -- plain, slow, single-threaded CPU oracle for lossless homomorphic
 * gradient compression (Count Sketch + bitmap index + peeling recovery).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The GPU library never
 * links, includes or calls it, and it shares no code with the GPU library.
 *
 * What it computes (paper sections cited per function in hco.c):
 *   Phase I   (Algorithm 1, sections 3.1, 3.2, 3.4): Count Sketch Y and bitmap B
 *             of one worker's gradient X.
 *   Aggregate (Algorithm 1, between the phases): Y <- sum of Y_w, B <- OR of B_w.
 *   Phase II  (Algorithm 1, section 3.2): synchronous peeling rounds, then the
 *             Count Sketch median estimate for whatever could not be peeled.
 *
 * Value types: int32 fixed point (sums wrap modulo 2^32, the way an integer
 * switch adds) and a floating-point path that the oracle runs in fp64.
 *
 * Sketch format (the paper fixes none of these details; the readings are
 * listed with the design notes of the repository):
 *   batch b = p / c, column t = p mod c             (section 3.4, c = 1024)
 *   h_j(b)  = SplitMix64 output number 3*b + j for state `seed`, j = 0, 1, 2
 *   rows    : r_0 = mulhi32(lo32(h_0), R)
 *             r_1 = mulhi32(lo32(h_1), R-1), then skip r_0
 *             r_2 = mulhi32(lo32(h_2), R-2), then skip min(r_0,r_1) and max(r_0,r_1)
 *             so the three rows of a batch are distinct (the three hash
 *             indexes of an element are different, section 3.1)
 *   bias_j  = (h_j >> 32) & (c - 1)                 (random rotation, section 3.4)
 *   g_j     = +1 if bit 63 of h_j is 0, else -1     (sign hash, section 3.1)
 *   cell_j(p) = r_j * c + ((t + bias_j) & (c - 1))
 *   B bit p = bit (p & 31) of 32-bit word p >> 5; bits past n are zero.
 *
 * Blocked sketch (section 3.2: the sketch split into blocks of a fixed size
 * so that peeling ends in O(1) rounds).  With block = K > 0 the batches are
 * grouped K at a time into parameter blocks q = b / K (the last one may be
 * shorter), and block q owns its own R_b = rows / nblocks consecutive rows:
 * the three rows above are drawn from R_b instead of R, sorted ascending and
 * offset by q * R_b.  An element's cells then all lie in its block's rows, so
 * the blocks peel independently.  The rotations of batch number i of block q
 * are bias_0 as above, bias_1 = bias_0 + (pi mod c), bias_2 = bias_0 +
 * (pi div c), mod c, with pi = P_q(i) a bijection of [0, c^2) keyed by
 * u_q = SplitMix64 output number 2^62 + q (see hco_batch_hash): two batches of
 * one block never share three rows with the same relative rotations
 * (c >= 32), which would put every pair of their corresponding elements on the
 * same three cells.  K * c must be a multiple of 32 (whole bitmap words per block).
 * block = 0 is the single global sketch (one block).
 *
 * Bloom-filter index (section 3.3), selected by bloom_k > 0: B is a bit array
 * of bloom_rows rows of c bits (the index reshaped into a matrix of width c,
 * section 3.4) instead of the bitmap.  Hash i < bloom_k of batch b is
 *   u_i(b) = SplitMix64 output number 3 * 2^32 + bloom_k * b + i for `seed`
 * (a counter range the sketch's outputs 3b + j, b < 2^32, never reach),
 *   brow_i = mulhi32(lo32(u_i), bloom_rows),  bbias_i = (u_i >> 32) & (c - 1),
 * and parameter p sets bit brow_i * c + ((t + bbias_i) & (c - 1)) for each i.
 * Bit q of the array is bit (q & 31) of word q >> 5; bits past
 * bloom_rows * c are zero.  A parameter is a candidate when all its bloom_k
 * bits are set: every nonzero is one, a zero is one with the filter's false
 * positive rate, and the decode peels the candidates (false positives are
 * recovered with value 0).
 */
#ifndef HCO_H
#define HCO_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    uint64_t n;     /* gradient length N, 1 .. 2^32-1                         */
    uint32_t k;     /* number of hashes; the paper uses three, only 3 accepted */
    uint32_t c;     /* batch width, power of two in [1, 1024]                 */
    uint64_t rows;  /* sketch rows R >= 3; cells = R * c < 2^32               */
    uint64_t seed;  /* hash seed shared by all workers                        */
    uint32_t block; /* batches per parameter block; 0 = one global sketch     */
    uint32_t bloom_k;     /* Bloom filter hashes (section 3.3); 0 = bitmap index */
    uint64_t bloom_rows;  /* rows of c bits in the Bloom filter (bloom_k > 0)    */
} hco_geom;

typedef struct {
    uint64_t n_support;    /* set bits of the aggregated bitmap                 */
    uint64_t n_recovered;  /* elements recovered by peeling                     */
    uint64_t rounds;       /* synchronous peeling rounds that peeled >= 1       */
    uint32_t success;      /* 1 iff every element of the support was peeled     */
    uint32_t pad;
} hco_info;

/* 0 on success, -1 on an invalid geometry. */
int hco_check_geom(const hco_geom *g);
/* rows = max(3, ceil(ceil(gamma * n_nonzero) / c)) -- sketch size >= gamma*n
 * (section 3.2, gamma = 1.23). */
uint64_t hco_rows_for(uint64_t n_nonzero, double gamma, uint32_t c);

/* Blocked sizing (a reading; the paper fixes only that blocks have a fixed
 * size): every block has block_rows rows; a block holds
 * K = floor(block_rows * n / (gamma * n_nonzero)) batches, clamped to
 * [1, min(max_block, batches)], so that its expected share of the support
 * times gamma fills its rows, then rounded down to a multiple of
 * max(1, 32 / c) so that a block holds whole bitmap words; R_b is
 * rows_for(the expected share of a block of K batches), at most block_rows.
 * Writes *block = K and *rows = nblocks * R_b.  Returns 0, or -1 on invalid
 * arguments. */
int hco_blocked_geometry(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                         uint32_t block_rows, uint32_t max_block, uint32_t *block,
                         uint64_t *rows);
/* Bloom sizing (section 3.3).  With lambda = (n - n_nonzero) / n_nonzero zero
 * parameters per nonzero and bit width `bits` (32 here), the false positive
 * rate is eps = 1 / (ln^2(2) * gamma * bits * lambda); the filter uses
 * k = max(1, round(log2(1 / eps))) hashes and k * n_nonzero / ln 2 bits
 * (so that half its bits are set and its false positive rate is 2^-k), in
 * whole rows of c bits; the sketch holds gamma * (n_nonzero + 2^-k * (n -
 * n_nonzero)) cells, the support plus the expected false positives, in whole
 * rows (at least three).  Writes *bloom_k, *bloom_rows, *rows and *eps (the
 * paper's eps before rounding).  Returns 0, or -1 on invalid arguments or when
 * k would round to zero (eps > 2^-1/2: the gradient is too dense for a filter
 * to pay). */
int hco_bloom_geometry(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                       uint32_t bits, uint32_t *bloom_k, uint64_t *bloom_rows,
                       uint64_t *rows, double *eps);
/* Words of the index B: ceil(n / 32) for the bitmap, ceil(bloom_rows * c / 32)
 * for a Bloom filter. */
uint64_t hco_index_words(const hco_geom *g);
/* The bloom_k bit positions of parameter p (bloom_k > 0). */
void hco_bloom_bits(const hco_geom *g, uint64_t p, uint64_t *bits);
/* Section 3.3 query for m parameters: out[i] = 1 iff all bloom_k bits of
 * idx[i] are set in the filter B. */
void hco_bloom_query(const hco_geom *g, const uint32_t *B, const uint64_t *idx, uint64_t m,
                     uint8_t *out);

/* Number of parameter blocks and rows per block of a geometry. */
uint64_t hco_nblocks(const hco_geom *g);
uint64_t hco_block_rows(const hco_geom *g);

/* SplitMix64: `count` consecutive outputs for state `seed`. */
void hco_splitmix64(uint64_t seed, uint64_t count, uint64_t *out);
/* rows, biases and signs of batch b. */
void hco_batch_hash(const hco_geom *g, uint64_t b, uint64_t row[3],
                    uint32_t bias[3], int32_t sign[3]);
/* cells[3*i+j], signs[3*i+j] for the parameters idx[0..m). */
void hco_cells(const hco_geom *g, const uint64_t *idx, uint64_t m,
               uint64_t *cells, int32_t *signs);

/* Phase I on a dense gradient.  Y[cells] and B[index words] are overwritten. */
int hco_encode_i32(const hco_geom *g, const int32_t *x, int32_t *Y, uint32_t *B);
int hco_encode_f64(const hco_geom *g, const double *x, double *Y, uint32_t *B);
/* Phase I on COO input (idx distinct, any order; zero values are skipped). */
int hco_encode_coo_i32(const hco_geom *g, const uint32_t *idx, const int32_t *val,
                       uint64_t nnz, int32_t *Y, uint32_t *B);
int hco_encode_coo_f64(const hco_geom *g, const uint32_t *idx, const double *val,
                       uint64_t nnz, double *Y, uint32_t *B);

/* Aggregation: Yout = sum over w of Yin[w] (int32 wraps; fp64 adds in worker
 * order 0..W-1), Bout = OR over w of Bin[w]. */
void hco_aggregate_i32(uint32_t W, uint64_t cells, uint64_t words,
                       const int32_t *Yin, const uint32_t *Bin,
                       int32_t *Yout, uint32_t *Bout);
void hco_aggregate_f64(uint32_t W, uint64_t cells, uint64_t words,
                       const double *Yin, const uint32_t *Bin,
                       double *Yout, uint32_t *Bout);

/* Phase II with synchronous rounds.  Y and B are not modified.
 * x_out[n]: recovered value, the median estimate for unpeeled members of the
 *           support, 0 outside the support.
 * mask[ceil(n/32)] (may be NULL): bit p set iff p was recovered by peeling.
 * round_of[n] (may be NULL): 1-based round that peeled p, 0 otherwise.
 * Returns 0, or -1 on an invalid geometry / allocation failure. */
int hco_decode_i32(const hco_geom *g, const int32_t *Y, const uint32_t *B,
                   int32_t *x_out, uint32_t *mask, hco_info *info,
                   uint32_t *round_of);
int hco_decode_f64(const hco_geom *g, const double *Y, const uint32_t *B,
                   double *x_out, uint32_t *mask, hco_info *info,
                   uint32_t *round_of);

/* Worst-case error propagation through the same synchronous schedule as
 * hco_decode_f64: given per-cell bounds dY[c] >= |error of Y[c]|, writes
 * bound[p] >= |error of the decoded x_p| for every p of the support (0 for
 * p outside it), valid for any rounding that stays within dY.  Peeling is
 * linear in Y for a fixed schedule: x = g_j * (Y[c] - sum of g' x' over the
 * earlier-peeled members of c), so |dx| <= dY[c] + sum of |dx'|; a leftover
 * estimate is a median, which moves by at most the largest of its three
 * cells' errors.  Section 3.2 does not fix which of an element's pure cells
 * supplies its value (in exact arithmetic they all hold it), so the bound of
 * a peeled element is the largest over all its cells pure in that round:
 * it holds whichever of them a decoder reads.  Returns 0 or -1. */
int hco_decode_bound_f64(const hco_geom *g, const double *dY, const uint32_t *B,
                         double *bound);

/* Independent cross-check: one-at-a-time peeling from a FIFO queue of pure
 * cells.  Same outputs as hco_decode_i32 except that info->rounds is 0. */
int hco_decode_queue_i32(const hco_geom *g, const int32_t *Y, const uint32_t *B,
                         int32_t *x_out, uint32_t *mask, hco_info *info);

/* Count Sketch query of section 3.1 for one parameter p: the median over j of
 * g_j(p) * Y[h_j(p)], on a sketch as given (no peeling). */
int32_t hco_query_i32(const hco_geom *g, const int32_t *Y, uint64_t p);
double  hco_query_f64(const hco_geom *g, const double *Y, uint64_t p);

/* Median of three (exposed for fixture tests of the estimator). */
int32_t hco_median3_i32(int32_t a, int32_t b, int32_t c);
double  hco_median3_f64(double a, double b, double c);

#ifdef __cplusplus
}
#endif
#endif
