/*
 * hco.c -- CPU oracle for lossless homomorphic gradient compression.
 *
 * TEST INFRASTRUCTURE ONLY (see hco.h).  Deliberately plain: no blocking, no
 * fusion, no threads.  Each function follows the paper's description in the
 * paper's order; the section each step comes from is named beside it.
 *
 * int32 arithmetic is done on uint32_t so that sums wrap modulo 2^32 without
 * undefined behaviour; the bit pattern is then read back as int32.
 */
#include "hco.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ hashing */

/* SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014; the finalizer constants are the ones of Vigna's
 * public-domain splitmix64.c).  Output i of state s is mix(s + (i+1)*golden). */
static uint64_t sm64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

static uint64_t sm64_output(uint64_t seed, uint64_t i)
{
    return sm64_mix(seed + (i + 1u) * 0x9e3779b97f4a7c15ULL);
}

void hco_splitmix64(uint64_t seed, uint64_t count, uint64_t *out)
{
    uint64_t state = seed;
    for (uint64_t i = 0; i < count; i++) {
        state += 0x9e3779b97f4a7c15ULL;
        out[i] = sm64_mix(state);
    }
}

/* floor(u * range / 2^32): maps a uniform 32-bit word to [0, range). */
static uint64_t scale32(uint64_t h, uint64_t range)
{
    return ((h & 0xffffffffULL) * range) >> 32;
}

uint64_t hco_nblocks(const hco_geom *g)
{
    if (g->block == 0) return 1;
    uint64_t batches = (g->n + g->c - 1) / g->c;
    return (batches + g->block - 1) / g->block;
}

uint64_t hco_block_rows(const hco_geom *g) { return g->rows / hco_nblocks(g); }

int hco_check_geom(const hco_geom *g)
{
    if (!g) return -1;
    if (g->k != 3) return -1;
    if (g->c == 0 || g->c > 1024 || (g->c & (g->c - 1)) != 0) return -1;
    if (g->n == 0 || g->n > 0xffffffffULL) return -1;
    if (g->rows < 3) return -1;
    if (g->rows > 0xffffffffULL / g->c) return -1; /* cells < 2^32 */
    if (g->block != 0) {
        /* every block owns the same whole number of rows, at least three */
        uint64_t nb = hco_nblocks(g);
        if (((uint64_t)g->block * g->c) % 32 != 0) return -1;
        if (g->rows % nb != 0 || g->rows / nb < 3) return -1;
    }
    if (g->bloom_k != 0) {
        /* a filter of bloom_rows rows of c bits, bit positions below 2^32 */
        if (g->bloom_k > 64 || g->bloom_rows == 0) return -1;
        if (g->bloom_rows > 0xffffffffULL / g->c) return -1;
    }
    return 0;
}

uint64_t hco_rows_for(uint64_t n_nonzero, double gamma, uint32_t c)
{
    /* sketch size at least gamma * n (section 3.2); whole rows of width c
     * (section 3.4); at least three rows so the three indexes can differ. */
    double need = gamma * (double)n_nonzero;
    uint64_t cells = (uint64_t)need;
    if ((double)cells < need) cells++;
    uint64_t rows = (cells + c - 1) / c;
    return rows < 3 ? 3 : rows;
}

int hco_blocked_geometry(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                         uint32_t block_rows, uint32_t max_block, uint32_t *block,
                         uint64_t *rows)
{
    if (n == 0 || n_nonzero == 0 || n_nonzero > n || !(gamma > 0.0)) return -1;
    if (c == 0 || c > 1024 || (c & (c - 1)) != 0 || block_rows < 3 || max_block == 0) return -1;
    uint64_t batches = (n + c - 1) / c;
    /* batches whose expected support times gamma fills block_rows rows */
    double k = floor((double)block_rows * (double)n / (gamma * (double)n_nonzero));
    uint64_t K = k < 1.0 ? 1 : (uint64_t)k;
    if (K > max_block) K = max_block;
    if (K > batches) K = batches;
    uint64_t unit = c >= 32 ? 1 : 32 / c; /* whole bitmap words per block */
    K -= K % unit;
    if (K == 0) K = unit;
    /* the expected support of a block of K batches, and the rows it needs */
    double share = (double)n_nonzero * (double)(K * c) / (double)n;
    uint64_t rb = hco_rows_for((uint64_t)ceil(share), gamma, c);
    if (rb > block_rows) rb = block_rows;
    uint64_t nblocks = (batches + K - 1) / K;
    *block = (uint32_t)K;
    *rows = nblocks * rb;
    return 0;
}

int hco_bloom_geometry(uint64_t n, uint64_t n_nonzero, double gamma, uint32_t c,
                       uint32_t bits, uint32_t *bloom_k, uint64_t *bloom_rows,
                       uint64_t *rows, double *eps)
{
    if (n == 0 || n_nonzero == 0 || n_nonzero >= n || !(gamma > 0.0) || bits == 0) return -1;
    if (c == 0 || c > 1024 || (c & (c - 1)) != 0) return -1;
    /* section 3.3: lambda * n zero parameters, eps = (ln^2 2 * gamma * C * lambda)^-1 */
    const double ln2 = log(2.0);
    double lambda = (double)(n - n_nonzero) / (double)n_nonzero;
    double e = 1.0 / (ln2 * ln2 * gamma * (double)bits * lambda);
    /* log(1/eps) hashes per nonzero; (n / ln 2) log(1/eps) bits */
    double k = floor(log2(1.0 / e) + 0.5);
    if (!(k >= 1.0)) return -1;
    if (k > 64.0) k = 64.0;
    double fbits = ceil(k * (double)n_nonzero / ln2);
    uint64_t brows = ((uint64_t)fbits + c - 1) / c;
    /* the sketch holds the candidates: the support and the zeros the filter
     * lets through, gamma * (n + eps (N - n)) cells (section 3.3's S_2) */
    double fp = ldexp(1.0, -(int)k);
    double cand = (double)n_nonzero + fp * (double)(n - n_nonzero);
    *bloom_k = (uint32_t)k;
    *bloom_rows = brows;
    *rows = hco_rows_for((uint64_t)ceil(cand), gamma, c);
    *eps = e;
    return 0;
}

uint64_t hco_index_words(const hco_geom *g)
{
    if (g->bloom_k == 0) return (g->n + 31) / 32;
    return (g->bloom_rows * g->c + 31) / 32;
}

/* Section 3.3: each nonzero is hashed to log(1/eps) bits of the filter;
 * section 3.4: the index is batched like the sketch, one row and one rotation
 * per batch and hash. */
void hco_bloom_bits(const hco_geom *g, uint64_t p, uint64_t *bits)
{
    uint64_t b = p / g->c, t = p % g->c;
    for (uint32_t i = 0; i < g->bloom_k; i++) {
        uint64_t u = sm64_output(g->seed, 3ULL * (1ULL << 32) + (uint64_t)g->bloom_k * b + i);
        uint64_t row = scale32(u, g->bloom_rows);
        uint64_t bias = (u >> 32) & (uint64_t)(g->c - 1);
        bits[i] = row * g->c + ((t + bias) % g->c);
    }
}

void hco_bloom_query(const hco_geom *g, const uint32_t *B, const uint64_t *idx, uint64_t m,
                     uint8_t *out)
{
    uint64_t bits[64];
    for (uint64_t e = 0; e < m; e++) {
        hco_bloom_bits(g, idx[e], bits);
        uint8_t all = 1;
        for (uint32_t i = 0; i < g->bloom_k; i++)
            if (!((B[bits[i] >> 5] >> (bits[i] & 31)) & 1u)) all = 0;
        out[e] = all;
    }
}

/* Section 3.1: three hash indexes and three signs per index; section 3.4: one
 * row index and one random rotation per batch of c parameters and per hash;
 * section 3.2: with a blocked sketch the rows come from the batch's block. */
void hco_batch_hash(const hco_geom *g, uint64_t b, uint64_t row[3],
                    uint32_t bias[3], int32_t sign[3])
{
    uint64_t h[3];
    for (int j = 0; j < 3; j++) h[j] = sm64_output(g->seed, 3u * b + (uint64_t)j);

    uint64_t R = g->block ? hco_block_rows(g) : g->rows;
    uint64_t base = g->block ? (b / g->block) * R : 0;
    uint64_t r0 = scale32(h[0], R);
    uint64_t r1 = scale32(h[1], R - 1);
    if (r1 >= r0) r1++;
    uint64_t lo = r0 < r1 ? r0 : r1;
    uint64_t hi = r0 < r1 ? r1 : r0;
    uint64_t r2 = scale32(h[2], R - 2);
    if (r2 >= lo) r2++;
    if (r2 >= hi) r2++;
    for (int j = 0; j < 3; j++) {
        bias[j] = (uint32_t)((h[j] >> 32) & (uint64_t)(g->c - 1));
        sign[j] = (h[j] >> 63) ? -1 : 1;
    }
    if (g->block == 0) {
        row[0] = r0;
        row[1] = r1;
        row[2] = r2;
        return;
    }
    /* blocked sketch: the three rows in ascending order, and the second and
     * third rotations offset from the first by the base-c digits of
     * pi = P(i), a bijection of [0, c^2) applied to the batch's index i in its
     * block and keyed by the block's constant u (SplitMix64 output 2^62 + q).
     * Distinct batches of a block then never share three rows with the same
     * relative rotations (c >= 32, so that c^2 >= 1024 >= K) -- a coincidence
     * that would put all their corresponding elements on the same three cells.
     * P: with M = c^2, a1, a2 and s the low, middle and high 20-bit fields of
     * u (a1, a2 made odd) and h = half the bits of M rounded up:
     * x = (i + s) mod M; x = x a1 mod M; x ^= x >> h; x = x a2 mod M; x ^= x >> h. */
    uint64_t v[3] = {r0, r1, r2};
    for (int x = 0; x < 2; x++)
        for (int y = 0; y < 2 - x; y++)
            if (v[y] > v[y + 1]) { uint64_t t = v[y]; v[y] = v[y + 1]; v[y + 1] = t; }
    for (int j = 0; j < 3; j++) row[j] = base + v[j];
    uint64_t q = b / g->block, i = b % g->block;
    uint64_t c = g->c, M = c * c;
    unsigned bits = 0;
    while ((1ULL << bits) < M) bits++;
    unsigned hshift = (bits + 1) / 2;
    uint64_t u = sm64_output(g->seed, (1ULL << 62) + q);
    uint64_t a1 = (u & 0xfffffULL) | 1ULL;
    uint64_t a2 = ((u >> 20) & 0xfffffULL) | 1ULL;
    uint64_t s0 = (u >> 40) & 0xfffffULL;
    uint64_t x = (i + s0) % M;
    x = (x * a1) % M;
    x ^= x >> hshift;
    x = (x * a2) % M;
    x ^= x >> hshift;
    bias[1] = (uint32_t)((bias[0] + x % c) % c);
    bias[2] = (uint32_t)((bias[0] + x / c) % c);
}

static uint64_t cell_of(const hco_geom *g, uint64_t p, const uint64_t row[3],
                        const uint32_t bias[3], int j)
{
    uint64_t t = p % g->c;
    return row[j] * g->c + ((t + bias[j]) % g->c);
}

void hco_cells(const hco_geom *g, const uint64_t *idx, uint64_t m,
               uint64_t *cells, int32_t *signs)
{
    for (uint64_t i = 0; i < m; i++) {
        uint64_t row[3];
        uint32_t bias[3];
        int32_t sign[3];
        hco_batch_hash(g, idx[i] / g->c, row, bias, sign);
        for (int j = 0; j < 3; j++) {
            cells[3 * i + j] = cell_of(g, idx[i], row, bias, j);
            signs[3 * i + j] = sign[j];
        }
    }
}

static uint64_t n_cells(const hco_geom *g) { return g->rows * g->c; }
static uint64_t n_words(const hco_geom *g) { return (g->n + 31) / 32; }

static void set_bit(uint32_t *B, uint64_t p) { B[p >> 5] |= 1u << (p & 31); }
static int get_bit(const uint32_t *B, uint64_t p) { return (B[p >> 5] >> (p & 31)) & 1u; }

/* Record nonzero parameter p in the index: its bit of the bitmap (section
 * 3.2), or its bloom_k bits of the Bloom filter (section 3.3). */
static void index_insert(const hco_geom *g, uint32_t *B, uint64_t p)
{
    if (g->bloom_k == 0) {
        set_bit(B, p);
        return;
    }
    uint64_t bits[64];
    hco_bloom_bits(g, p, bits);
    for (uint32_t i = 0; i < g->bloom_k; i++) set_bit(B, bits[i]);
}

/* The parameters the index reports as nonzero, as a bitmap of n bits: the
 * bitmap itself, or every p whose bloom_k filter bits are all set (the query
 * of section 3.3). */
static void index_support(const hco_geom *g, const uint32_t *B, uint32_t *out)
{
    memset(out, 0, n_words(g) * sizeof(uint32_t));
    for (uint64_t p = 0; p < g->n; p++) {
        int member;
        if (g->bloom_k == 0) {
            member = get_bit(B, p);
        } else {
            uint64_t bits[64];
            hco_bloom_bits(g, p, bits);
            member = 1;
            for (uint32_t i = 0; i < g->bloom_k; i++)
                if (!get_bit(B, bits[i])) member = 0;
        }
        if (member) set_bit(out, p);
    }
}

/* g * v with int32 wrap-around. */
static uint32_t signed_u32(int32_t sign, uint32_t v) { return sign < 0 ? 0u - v : v; }

/* ------------------------------------------------------------------- encode */

/* Algorithm 1 Phase I: build the Count Sketch Y (section 3.1: Y[h_j(i)] +=
 * g_j(i) * x_i for j = 1..3, batched as in section 3.4) and the bitmap index B
 * (section 3.2: one bit per parameter, set iff the parameter is nonzero). */
int hco_encode_i32(const hco_geom *g, const int32_t *x, int32_t *Y, uint32_t *B)
{
    if (hco_check_geom(g)) return -1;
    uint32_t *Yu = (uint32_t *)Y;
    memset(Y, 0, n_cells(g) * sizeof(int32_t));
    memset(B, 0, hco_index_words(g) * sizeof(uint32_t));
    for (uint64_t p = 0; p < g->n; p++) {
        if (x[p] == 0) continue;
        index_insert(g, B, p);
        uint64_t row[3];
        uint32_t bias[3];
        int32_t sign[3];
        hco_batch_hash(g, p / g->c, row, bias, sign);
        for (int j = 0; j < 3; j++)
            Yu[cell_of(g, p, row, bias, j)] += signed_u32(sign[j], (uint32_t)x[p]);
    }
    return 0;
}

int hco_encode_f64(const hco_geom *g, const double *x, double *Y, uint32_t *B)
{
    if (hco_check_geom(g)) return -1;
    memset(B, 0, hco_index_words(g) * sizeof(uint32_t));
    for (uint64_t i = 0; i < n_cells(g); i++) Y[i] = 0.0;
    for (uint64_t p = 0; p < g->n; p++) {
        if (x[p] == 0.0) continue;
        index_insert(g, B, p);
        uint64_t row[3];
        uint32_t bias[3];
        int32_t sign[3];
        hco_batch_hash(g, p / g->c, row, bias, sign);
        for (int j = 0; j < 3; j++) Y[cell_of(g, p, row, bias, j)] += sign[j] * x[p];
    }
    return 0;
}

int hco_encode_coo_i32(const hco_geom *g, const uint32_t *idx, const int32_t *val,
                       uint64_t nnz, int32_t *Y, uint32_t *B)
{
    if (hco_check_geom(g)) return -1;
    uint32_t *Yu = (uint32_t *)Y;
    memset(Y, 0, n_cells(g) * sizeof(int32_t));
    memset(B, 0, hco_index_words(g) * sizeof(uint32_t));
    for (uint64_t e = 0; e < nnz; e++) {
        uint64_t p = idx[e];
        if (p >= g->n) return -1;
        if (val[e] == 0) continue;
        index_insert(g, B, p);
        uint64_t row[3];
        uint32_t bias[3];
        int32_t sign[3];
        hco_batch_hash(g, p / g->c, row, bias, sign);
        for (int j = 0; j < 3; j++)
            Yu[cell_of(g, p, row, bias, j)] += signed_u32(sign[j], (uint32_t)val[e]);
    }
    return 0;
}

int hco_encode_coo_f64(const hco_geom *g, const uint32_t *idx, const double *val,
                       uint64_t nnz, double *Y, uint32_t *B)
{
    if (hco_check_geom(g)) return -1;
    memset(B, 0, hco_index_words(g) * sizeof(uint32_t));
    for (uint64_t i = 0; i < n_cells(g); i++) Y[i] = 0.0;
    for (uint64_t e = 0; e < nnz; e++) {
        uint64_t p = idx[e];
        if (p >= g->n) return -1;
        if (val[e] == 0.0) continue;
        index_insert(g, B, p);
        uint64_t row[3];
        uint32_t bias[3];
        int32_t sign[3];
        hco_batch_hash(g, p / g->c, row, bias, sign);
        for (int j = 0; j < 3; j++) Y[cell_of(g, p, row, bias, j)] += sign[j] * val[e];
    }
    return 0;
}

/* ---------------------------------------------------------------- aggregate */

/* What the aggregation API does between the two phases of Algorithm 1:
 * Y <- sum of Y (arithmetic sum), B <- OR of B (section 3.2). */
void hco_aggregate_i32(uint32_t W, uint64_t cells, uint64_t words,
                       const int32_t *Yin, const uint32_t *Bin,
                       int32_t *Yout, uint32_t *Bout)
{
    for (uint64_t i = 0; i < cells; i++) {
        uint32_t s = 0;
        for (uint32_t w = 0; w < W; w++) s += (uint32_t)Yin[(uint64_t)w * cells + i];
        Yout[i] = (int32_t)s;
    }
    for (uint64_t i = 0; i < words; i++) {
        uint32_t o = 0;
        for (uint32_t w = 0; w < W; w++) o |= Bin[(uint64_t)w * words + i];
        Bout[i] = o;
    }
}

void hco_aggregate_f64(uint32_t W, uint64_t cells, uint64_t words,
                       const double *Yin, const uint32_t *Bin,
                       double *Yout, uint32_t *Bout)
{
    for (uint64_t i = 0; i < cells; i++) {
        double s = 0.0;
        for (uint32_t w = 0; w < W; w++) s += Yin[(uint64_t)w * cells + i];
        Yout[i] = s;
    }
    for (uint64_t i = 0; i < words; i++) {
        uint32_t o = 0;
        for (uint32_t w = 0; w < W; w++) o |= Bin[(uint64_t)w * words + i];
        Bout[i] = o;
    }
}

/* ------------------------------------------------------------------- decode */

int32_t hco_median3_i32(int32_t a, int32_t b, int32_t c)
{
    int32_t t;
    if (a > b) { t = a; a = b; b = t; }
    if (b > c) { t = b; b = c; c = t; }
    if (a > b) { t = a; a = b; b = t; }
    return b;
}

double hco_median3_f64(double a, double b, double c)
{
    double t;
    if (a > b) { t = a; a = b; b = t; }
    if (b > c) { t = b; b = c; c = t; }
    if (a > b) { t = a; a = b; b = t; }
    return b;
}

/* Section 3.1: the estimate of x_p is the median over j of g_j(p) * Y[h_j(p)]. */
int32_t hco_query_i32(const hco_geom *g, const int32_t *Y, uint64_t p)
{
    uint64_t row[3];
    uint32_t bias[3];
    int32_t sign[3];
    hco_batch_hash(g, p / g->c, row, bias, sign);
    int32_t v[3];
    for (int j = 0; j < 3; j++)
        v[j] = (int32_t)signed_u32(sign[j], (uint32_t)Y[cell_of(g, p, row, bias, j)]);
    return hco_median3_i32(v[0], v[1], v[2]);
}

double hco_query_f64(const hco_geom *g, const double *Y, uint64_t p)
{
    uint64_t row[3];
    uint32_t bias[3];
    int32_t sign[3];
    hco_batch_hash(g, p / g->c, row, bias, sign);
    double v[3];
    for (int j = 0; j < 3; j++) v[j] = sign[j] * Y[cell_of(g, p, row, bias, j)];
    return hco_median3_f64(v[0], v[1], v[2]);
}

/* The candidate bitmap of an index (index_support) in a new allocation, or
 * NULL if out of memory. */
static uint32_t *candidates(const hco_geom *g, const uint32_t *B)
{
    uint32_t *cand = (uint32_t *)malloc(n_words(g) * sizeof(uint32_t));
    if (cand) index_support(g, B, cand);
    return cand;
}

/* The support (set bits of B) as an ascending list with each element's three
 * cells and signs.  Returns the element count, or UINT64_MAX on allocation
 * failure (*out_* are then NULL). */
static uint64_t support_of(const hco_geom *g, const uint32_t *B, uint64_t **out_p,
                           uint64_t **out_cell, int32_t **out_sign)
{
    uint64_t m = 0;
    for (uint64_t p = 0; p < g->n; p++) m += (uint64_t)get_bit(B, p);
    uint64_t *ps = (uint64_t *)malloc((m ? m : 1) * sizeof(uint64_t));
    uint64_t *cell = (uint64_t *)malloc((m ? m : 1) * 3 * sizeof(uint64_t));
    int32_t *sign = (int32_t *)malloc((m ? m : 1) * 3 * sizeof(int32_t));
    if (!ps || !cell || !sign) {
        free(ps); free(cell); free(sign);
        *out_p = NULL; *out_cell = NULL; *out_sign = NULL;
        return UINT64_MAX;
    }
    uint64_t i = 0;
    for (uint64_t p = 0; p < g->n; p++)
        if (get_bit(B, p)) ps[i++] = p;
    hco_cells(g, ps, m, cell, sign);
    *out_p = ps;
    *out_cell = cell;
    *out_sign = sign;
    return m;
}

/* Algorithm 1 Phase II with the peeling of section 3.2, run as synchronous
 * rounds (the parallel peeling the section cites).  In each round:
 *   1. from the bitmap of parameters not yet recovered, find the sketch cells
 *      that exactly one such parameter maps to;
 *   2. every parameter owning such a cell is recovered from it, x = g_j * Y
 *      (when several of its cells qualify, the one with the smallest j);
 *   3. each recovered parameter is cleared from the bitmap and deducted from
 *      all three of its cells, Y[h_j] -= g_j * x.
 * Rounds stop when a round recovers nothing.  Parameters still set in the
 * bitmap get the Count Sketch median estimate from the residual sketch
 * (the last recovery step of Algorithm 1; footnote of 3.2). */
int hco_decode_i32(const hco_geom *g, const int32_t *Y, const uint32_t *B,
                   int32_t *x_out, uint32_t *mask, hco_info *info,
                   uint32_t *round_of)
{
    if (hco_check_geom(g)) return -1;
    const uint64_t C = n_cells(g);
    uint64_t *ps, *cell;
    int32_t *sign;
    uint32_t *cand = candidates(g, B);
    if (!cand) return -1;
    const uint64_t m = support_of(g, cand, &ps, &cell, &sign);
    if (m == UINT64_MAX) { free(cand); return -1; }

    uint32_t *Yr = (uint32_t *)malloc(C * sizeof(uint32_t));       /* residual sketch */
    uint32_t *bits = (uint32_t *)malloc(n_words(g) * sizeof(uint32_t)); /* working bitmap */
    uint32_t *deg = (uint32_t *)malloc(C * sizeof(uint32_t));
    uint32_t *val = (uint32_t *)malloc((m ? m : 1) * sizeof(uint32_t));
    int8_t *pick = (int8_t *)malloc(m ? m : 1); /* j of the pure cell, or -1 */
    if (!Yr || !bits || !deg || !val || !pick) {
        free(Yr); free(bits); free(deg); free(val); free(pick);
        free(ps); free(cell); free(sign); free(cand);
        return -1;
    }
    memcpy(Yr, Y, C * sizeof(uint32_t));
    memcpy(bits, cand, n_words(g) * sizeof(uint32_t));
    memset(x_out, 0, g->n * sizeof(int32_t));
    if (mask) memset(mask, 0, n_words(g) * sizeof(uint32_t));
    if (round_of) memset(round_of, 0, g->n * sizeof(uint32_t));

    uint64_t rounds = 0, recovered = 0;
    for (;;) {
        /* 1. cells mapped by exactly one parameter still in the bitmap */
        memset(deg, 0, C * sizeof(uint32_t));
        for (uint64_t i = 0; i < m; i++)
            if (get_bit(bits, ps[i]))
                for (int j = 0; j < 3; j++) deg[cell[3 * i + j]]++;

        /* 2. parameters that own such a cell, valued from it */
        uint64_t peeled = 0;
        for (uint64_t i = 0; i < m; i++) {
            pick[i] = -1;
            if (!get_bit(bits, ps[i])) continue;
            for (int j = 0; j < 3; j++) {
                if (deg[cell[3 * i + j]] == 1) {
                    pick[i] = (int8_t)j;
                    val[i] = signed_u32(sign[3 * i + j], Yr[cell[3 * i + j]]);
                    peeled++;
                    break;
                }
            }
        }
        if (peeled == 0) break;
        rounds++;

        /* 3. clear from the bitmap and deduct from the sketch */
        for (uint64_t i = 0; i < m; i++) {
            if (pick[i] < 0) continue;
            bits[ps[i] >> 5] &= ~(1u << (ps[i] & 31));
            for (int j = 0; j < 3; j++)
                Yr[cell[3 * i + j]] -= signed_u32(sign[3 * i + j], val[i]);
            x_out[ps[i]] = (int32_t)val[i];
            if (mask) set_bit(mask, ps[i]);
            if (round_of) round_of[ps[i]] = (uint32_t)rounds;
            recovered++;
        }
    }

    /* leftovers: Count Sketch estimate on the residual sketch */
    for (uint64_t i = 0; i < m; i++) {
        if (!get_bit(bits, ps[i])) continue;
        int32_t v[3];
        for (int j = 0; j < 3; j++)
            v[j] = (int32_t)signed_u32(sign[3 * i + j], Yr[cell[3 * i + j]]);
        x_out[ps[i]] = hco_median3_i32(v[0], v[1], v[2]);
    }

    if (info) {
        info->n_support = m;
        info->n_recovered = recovered;
        info->rounds = rounds;
        info->success = recovered == m;
        info->pad = 0;
    }
    free(Yr); free(bits); free(deg); free(val); free(pick);
    free(ps); free(cell); free(sign); free(cand);
    return 0;
}

int hco_decode_f64(const hco_geom *g, const double *Y, const uint32_t *B,
                   double *x_out, uint32_t *mask, hco_info *info,
                   uint32_t *round_of)
{
    if (hco_check_geom(g)) return -1;
    const uint64_t C = n_cells(g);
    uint64_t *ps, *cell;
    int32_t *sign;
    uint32_t *cand = candidates(g, B);
    if (!cand) return -1;
    const uint64_t m = support_of(g, cand, &ps, &cell, &sign);
    if (m == UINT64_MAX) { free(cand); return -1; }

    double *Yr = (double *)malloc(C * sizeof(double));
    uint32_t *bits = (uint32_t *)malloc(n_words(g) * sizeof(uint32_t));
    uint32_t *deg = (uint32_t *)malloc(C * sizeof(uint32_t));
    double *val = (double *)malloc((m ? m : 1) * sizeof(double));
    int8_t *pick = (int8_t *)malloc(m ? m : 1);
    if (!Yr || !bits || !deg || !val || !pick) {
        free(Yr); free(bits); free(deg); free(val); free(pick);
        free(ps); free(cell); free(sign); free(cand);
        return -1;
    }
    memcpy(Yr, Y, C * sizeof(double));
    memcpy(bits, cand, n_words(g) * sizeof(uint32_t));
    for (uint64_t p = 0; p < g->n; p++) x_out[p] = 0.0;
    if (mask) memset(mask, 0, n_words(g) * sizeof(uint32_t));
    if (round_of) memset(round_of, 0, g->n * sizeof(uint32_t));

    uint64_t rounds = 0, recovered = 0;
    for (;;) {
        memset(deg, 0, C * sizeof(uint32_t));
        for (uint64_t i = 0; i < m; i++)
            if (get_bit(bits, ps[i]))
                for (int j = 0; j < 3; j++) deg[cell[3 * i + j]]++;

        uint64_t peeled = 0;
        for (uint64_t i = 0; i < m; i++) {
            pick[i] = -1;
            if (!get_bit(bits, ps[i])) continue;
            for (int j = 0; j < 3; j++) {
                if (deg[cell[3 * i + j]] == 1) {
                    pick[i] = (int8_t)j;
                    val[i] = sign[3 * i + j] * Yr[cell[3 * i + j]];
                    peeled++;
                    break;
                }
            }
        }
        if (peeled == 0) break;
        rounds++;

        for (uint64_t i = 0; i < m; i++) {
            if (pick[i] < 0) continue;
            bits[ps[i] >> 5] &= ~(1u << (ps[i] & 31));
            for (int j = 0; j < 3; j++) Yr[cell[3 * i + j]] -= sign[3 * i + j] * val[i];
            x_out[ps[i]] = val[i];
            if (mask) set_bit(mask, ps[i]);
            if (round_of) round_of[ps[i]] = (uint32_t)rounds;
            recovered++;
        }
    }

    for (uint64_t i = 0; i < m; i++) {
        if (!get_bit(bits, ps[i])) continue;
        double v[3];
        for (int j = 0; j < 3; j++) v[j] = sign[3 * i + j] * Yr[cell[3 * i + j]];
        x_out[ps[i]] = hco_median3_f64(v[0], v[1], v[2]);
    }

    if (info) {
        info->n_support = m;
        info->n_recovered = recovered;
        info->rounds = rounds;
        info->success = recovered == m;
        info->pad = 0;
    }
    free(Yr); free(bits); free(deg); free(val); free(pick);
    free(ps); free(cell); free(sign); free(cand);
    return 0;
}

/* Error bound carried through the schedule of hco_decode_f64 (see hco.h).
 * The schedule (which cells are pure in which round) depends only on B and
 * the hashes, so this repeats it with absolute-value accumulation in place
 * of subtraction, taking for each peeled element the largest bound among its
 * pure cells. */
int hco_decode_bound_f64(const hco_geom *g, const double *dY, const uint32_t *B,
                         double *bound)
{
    if (hco_check_geom(g)) return -1;
    const uint64_t C = n_cells(g);
    uint64_t *ps, *cell;
    int32_t *sign;
    uint32_t *cand = candidates(g, B);
    if (!cand) return -1;
    const uint64_t m = support_of(g, cand, &ps, &cell, &sign);
    if (m == UINT64_MAX) { free(cand); return -1; }

    double *Eb = (double *)malloc(C * sizeof(double));    /* accumulated cell error */
    uint32_t *bits = (uint32_t *)malloc(n_words(g) * sizeof(uint32_t));
    uint32_t *deg = (uint32_t *)malloc(C * sizeof(uint32_t));
    double *eb = (double *)malloc((m ? m : 1) * sizeof(double));
    int8_t *pick = (int8_t *)malloc(m ? m : 1);
    if (!Eb || !bits || !deg || !eb || !pick) {
        free(Eb); free(bits); free(deg); free(eb); free(pick);
        free(ps); free(cell); free(sign); free(cand);
        return -1;
    }
    for (uint64_t i = 0; i < C; i++) Eb[i] = dY[i] < 0 ? -dY[i] : dY[i];
    memcpy(bits, cand, n_words(g) * sizeof(uint32_t));
    for (uint64_t p = 0; p < g->n; p++) bound[p] = 0.0;

    for (;;) {
        memset(deg, 0, C * sizeof(uint32_t));
        for (uint64_t i = 0; i < m; i++)
            if (get_bit(bits, ps[i]))
                for (int j = 0; j < 3; j++) deg[cell[3 * i + j]]++;
        uint64_t peeled = 0;
        for (uint64_t i = 0; i < m; i++) {
            pick[i] = -1;
            if (!get_bit(bits, ps[i])) continue;
            for (int j = 0; j < 3; j++) {
                if (deg[cell[3 * i + j]] != 1) continue;
                if (pick[i] < 0) {
                    pick[i] = (int8_t)j;
                    eb[i] = Eb[cell[3 * i + j]];
                    peeled++;
                } else if (Eb[cell[3 * i + j]] > eb[i]) {
                    eb[i] = Eb[cell[3 * i + j]];
                }
            }
        }
        if (peeled == 0) break;
        for (uint64_t i = 0; i < m; i++) {
            if (pick[i] < 0) continue;
            bits[ps[i] >> 5] &= ~(1u << (ps[i] & 31));
            for (int j = 0; j < 3; j++) Eb[cell[3 * i + j]] += eb[i];
            bound[ps[i]] = eb[i];
        }
    }
    for (uint64_t i = 0; i < m; i++) {
        if (!get_bit(bits, ps[i])) continue;
        double b = 0.0;
        for (int j = 0; j < 3; j++)
            if (Eb[cell[3 * i + j]] > b) b = Eb[cell[3 * i + j]];
        bound[ps[i]] = b;
    }
    free(Eb); free(bits); free(deg); free(eb); free(pick);
    free(ps); free(cell); free(sign); free(cand);
    return 0;
}

/* Sequential peeling, one parameter at a time, driven by a FIFO queue of cells
 * that exactly one live parameter maps to (the classic peeling the parallel
 * version speeds up).  Written independently of hco_decode_i32 so the two can
 * check each other: the peeled set (the complement of the 2-core) and the
 * int32 values must agree. */
int hco_decode_queue_i32(const hco_geom *g, const int32_t *Y, const uint32_t *B,
                         int32_t *x_out, uint32_t *mask, hco_info *info)
{
    if (hco_check_geom(g)) return -1;
    const uint64_t C = n_cells(g);
    uint64_t *ps, *cell;
    int32_t *sign;
    uint32_t *cand = candidates(g, B);
    if (!cand) return -1;
    const uint64_t m = support_of(g, cand, &ps, &cell, &sign);
    if (m == UINT64_MAX) { free(cand); return -1; }

    uint32_t *Yr = (uint32_t *)malloc(C * sizeof(uint32_t));
    uint64_t *deg = (uint64_t *)calloc(C, sizeof(uint64_t));
    uint64_t *start = (uint64_t *)calloc(C + 1, sizeof(uint64_t));
    uint64_t *fill = (uint64_t *)calloc(C, sizeof(uint64_t));
    uint64_t *adj = (uint64_t *)malloc((m ? 3 * m : 1) * sizeof(uint64_t));
    uint8_t *alive = (uint8_t *)malloc(m ? m : 1);
    uint64_t *queue = (uint64_t *)malloc((3 * m + C + 1) * sizeof(uint64_t));
    if (!Yr || !deg || !start || !fill || !adj || !alive || !queue) {
        free(Yr); free(deg); free(start); free(fill); free(adj); free(alive); free(queue);
        free(ps); free(cell); free(sign); free(cand);
        return -1;
    }
    memcpy(Yr, Y, C * sizeof(uint32_t));
    memset(x_out, 0, g->n * sizeof(int32_t));
    if (mask) memset(mask, 0, n_words(g) * sizeof(uint32_t));

    /* cell -> incident elements, as a compressed adjacency list */
    for (uint64_t i = 0; i < 3 * m; i++) deg[cell[i]]++;
    for (uint64_t cc = 0; cc < C; cc++) start[cc + 1] = start[cc] + deg[cc];
    for (uint64_t i = 0; i < 3 * m; i++) adj[start[cell[i]] + fill[cell[i]]++] = i / 3;
    for (uint64_t i = 0; i < m; i++) alive[i] = 1;

    uint64_t qh = 0, qt = 0, recovered = 0;
    for (uint64_t cc = 0; cc < C; cc++)
        if (deg[cc] == 1) queue[qt++] = cc;
    while (qh < qt) {
        uint64_t cc = queue[qh++];
        if (deg[cc] != 1) continue;
        uint64_t e = UINT64_MAX;
        for (uint64_t a = start[cc]; a < start[cc + 1]; a++)
            if (alive[adj[a]]) { e = adj[a]; break; }
        if (e == UINT64_MAX) continue;
        int jj = 0;
        while (cell[3 * e + jj] != cc) jj++;
        uint32_t v = signed_u32(sign[3 * e + jj], Yr[cc]);
        alive[e] = 0;
        recovered++;
        x_out[ps[e]] = (int32_t)v;
        if (mask) set_bit(mask, ps[e]);
        for (int j = 0; j < 3; j++) {
            uint64_t d = cell[3 * e + j];
            Yr[d] -= signed_u32(sign[3 * e + j], v);
            deg[d]--;
            if (deg[d] == 1) queue[qt++] = d;
        }
    }

    for (uint64_t i = 0; i < m; i++) {
        if (!alive[i]) continue;
        int32_t v[3];
        for (int j = 0; j < 3; j++)
            v[j] = (int32_t)signed_u32(sign[3 * i + j], Yr[cell[3 * i + j]]);
        x_out[ps[i]] = hco_median3_i32(v[0], v[1], v[2]);
    }
    if (info) {
        info->n_support = m;
        info->n_recovered = recovered;
        info->rounds = 0;
        info->success = recovered == m;
        info->pad = 0;
    }
    free(Yr); free(deg); free(start); free(fill); free(adj); free(alive); free(queue);
    free(ps); free(cell); free(sign); free(cand);
    return 0;
}
