/*
 * DARB CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously-correct C reference for the DARB hot path
 * (Ren et al., "DARB: A Density-Adaptive Regular-Block Pruning for Deep
 * Neural Networks", AAAI-20).  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this code; the product library never
 * does, and the two share no source.
 *
 * What it computes, in the paper's order:
 *   1. block size per row from the row density (section 3.2, the rounding rule
 *      with its worked example; the "floor" variant always rounds the density
 *      up to the next power-of-two fraction);
 *   2. the storage layout: rows grouped by block size (section 3.2, the
 *      power-of-two density groups that make storage regular), ceil(N/b)
 *      blocks per row (section 4.2 / Table 7 fix the partial tail block);
 *   3. block-max weight masking (section 3.1, BMWM: split a row into equal
 *      blocks, keep the largest-magnitude weight of each block, repeat per row);
 *   4. decode to the masked dense matrix;
 *   5. the product with the retained weights only (section 2: pruned weights are
 *      neither stored nor computed; section 3.2: each block's in-block index
 *      selects one activation), accumulated in fp64.
 *
 * Readings where the paper is silent (all listed in the design notes):
 *   - a row of density exactly D rounds up (like the denser rows);
 *   - a row of density 0 gets the largest allowed block size;
 *   - "largest magnitude" is decided on the stored bits with the sign cleared,
 *     compared as unsigned integers; equal keys go to the lowest in-block index;
 *   - a tail block shorter than b only offers its in-range elements.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_EFORMAT (-2)

enum { ROUND_FLOOR = 0, ROUND_PAPER = 1 };
enum { DT_F32 = 0, DT_F16 = 1 };

static int is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

static int ilog2(int64_t v) {
    int l = 0;
    while (((int64_t)1 << l) < v) ++l;
    return l;
}

/* IEEE-754 binary16 -> double, from the format's definition. */
double oracle_half_to_double(uint16_t h) {
    int s = (h >> 15) & 1;
    int e = (h >> 10) & 0x1F;
    int m = h & 0x3FF;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24);                 /* subnormal: m * 2^-24 */
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(m | 0x400), e - 25);    /* 1.m * 2^(e-15) */
    return s ? -v : v;
}

static double f32_bits_to_double(uint32_t u) {
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * Step 1: block size of every row (section 3.2).
 *
 * A row of density d is given block size b = 1/d', where d' is d moved to a
 * power-of-two fraction.  f below is the largest power of two with f*d <= 1,
 * so 1/f is d rounded up; 1/(2f) (or 1/f when f*d == 1) is d rounded down.
 * Paper mode rounds up when d >= D and down when d < D; floor mode always
 * rounds up.  Products with a power of two are exact in fp64, so every
 * comparison here is exact.  The result is clamped to [b_min, b_max].
 */
int oracle_block_log2(int64_t M, const double *row_density, double matrix_density,
                      int mode, int b_min, int b_max, uint8_t *log2b) {
    if (M < 0 || (M > 0 && (!row_density || !log2b))) return ORACLE_EINVAL;
    if (!is_pow2(b_min) || !is_pow2(b_max) || b_min > b_max || b_max > 128) return ORACLE_EINVAL;
    if (mode != ROUND_FLOOR && mode != ROUND_PAPER) return ORACLE_EINVAL;
    if (!(matrix_density >= 0.0 && matrix_density <= 1.0)) return ORACLE_EINVAL;
    for (int64_t r = 0; r < M; ++r) {
        double d = row_density[r];
        if (!(d >= 0.0 && d <= 1.0)) return ORACLE_EINVAL;
    }
    for (int64_t r = 0; r < M; ++r) {
        double d = row_density[r];
        double b;
        if (d == 0.0) {
            b = (double)b_max;
        } else {
            double f = 1.0;
            while (2.0 * f * d <= 1.0) f *= 2.0;
            if (mode == ROUND_FLOOR || d >= matrix_density)
                b = f;                                  /* density rounded up   */
            else
                b = (f * d == 1.0) ? f : 2.0 * f;       /* density rounded down */
        }
        if (b < (double)b_min) b = (double)b_min;
        if (b > (double)b_max) b = (double)b_max;
        log2b[r] = (uint8_t)ilog2((int64_t)b);
    }
    return ORACLE_OK;
}

/*
 * Step 2: storage layout.  Rows are grouped by block size, smallest block size
 * first; inside a group rows keep their original order; a row of block size b
 * owns ceil(N/b) consecutive slots.  perm[i] is the original row stored i-th,
 * row_start[r] the first slot of row r.  Returns the retained-weight count.
 */
int64_t oracle_layout(int64_t M, int64_t N, const uint8_t *log2b, int32_t *perm,
                      int64_t *row_start) {
    if (M < 0 || N <= 0) return ORACLE_EINVAL;
    int64_t pos = 0, i = 0;
    for (int l = 0; l <= 7; ++l) {
        int64_t b = (int64_t)1 << l;
        for (int64_t r = 0; r < M; ++r) {
            if (log2b[r] != l) continue;
            perm[i++] = (int32_t)r;
            row_start[r] = pos;
            pos += (N + b - 1) / b;
        }
    }
    if (i != M) return ORACLE_EINVAL;   /* some log2b > 7 */
    return pos;
}

/*
 * Step 3: block-max weight masking (section 3.1).  For every row r and block k
 * the candidates are columns k*b + j, j < b, that lie inside the row.  The kept
 * element is the first one whose magnitude key is the block's maximum.  The
 * kept value is copied bit for bit, its in-block index j is the offset.
 */
void oracle_encode_f32(int64_t M, int64_t N, const uint32_t *W, int64_t ldw,
                       const uint8_t *log2b, const int64_t *row_start,
                       uint32_t *values, uint8_t *offsets) {
    for (int64_t r = 0; r < M; ++r) {
        int64_t b = (int64_t)1 << log2b[r];
        int64_t nblk = (N + b - 1) / b;
        const uint32_t *row = W + r * ldw;
        for (int64_t k = 0; k < nblk; ++k) {
            int64_t best = 0;
            uint32_t best_key = row[k * b] & 0x7FFFFFFFu;
            for (int64_t j = 1; j < b && k * b + j < N; ++j) {
                uint32_t key = row[k * b + j] & 0x7FFFFFFFu;
                if (key > best_key) { best_key = key; best = j; }
            }
            values[row_start[r] + k] = row[k * b + best];
            offsets[row_start[r] + k] = (uint8_t)best;
        }
    }
}

void oracle_encode_f16(int64_t M, int64_t N, const uint16_t *W, int64_t ldw,
                       const uint8_t *log2b, const int64_t *row_start,
                       uint16_t *values, uint8_t *offsets) {
    for (int64_t r = 0; r < M; ++r) {
        int64_t b = (int64_t)1 << log2b[r];
        int64_t nblk = (N + b - 1) / b;
        const uint16_t *row = W + r * ldw;
        for (int64_t k = 0; k < nblk; ++k) {
            int64_t best = 0;
            uint16_t best_key = row[k * b] & 0x7FFFu;
            for (int64_t j = 1; j < b && k * b + j < N; ++j) {
                uint16_t key = row[k * b + j] & 0x7FFFu;
                if (key > best_key) { best_key = key; best = j; }
            }
            values[row_start[r] + k] = row[k * b + best];
            offsets[row_start[r] + k] = (uint8_t)best;
        }
    }
}

/*
 * Step 4: decode into the masked dense matrix: +0.0 everywhere except the kept
 * positions, which receive the kept bits.  elem_bytes is 4 (fp32) or 2 (fp16).
 * Returns ORACLE_EFORMAT if an offset points outside its block or the row.
 */
int oracle_decode(int64_t M, int64_t N, int elem_bytes, const void *values,
                  const uint8_t *offsets, const uint8_t *log2b, const int64_t *row_start,
                  void *Wout, int64_t ldw) {
    for (int64_t r = 0; r < M; ++r) {
        int64_t b = (int64_t)1 << log2b[r];
        int64_t nblk = (N + b - 1) / b;
        for (int64_t c = 0; c < N; ++c) {
            if (elem_bytes == 4) ((uint32_t *)Wout)[r * ldw + c] = 0u;
            else ((uint16_t *)Wout)[r * ldw + c] = 0u;
        }
        for (int64_t k = 0; k < nblk; ++k) {
            int64_t s = row_start[r] + k;
            int64_t c = k * b + offsets[s];
            if (offsets[s] >= b || c >= N) return ORACLE_EFORMAT;
            if (elem_bytes == 4) ((uint32_t *)Wout)[r * ldw + c] = ((const uint32_t *)values)[s];
            else ((uint16_t *)Wout)[r * ldw + c] = ((const uint16_t *)values)[s];
        }
    }
    return ORACLE_OK;
}

static double load_elem(int dtype, const void *p, int64_t i) {
    if (dtype == DT_F32) return f32_bits_to_double(((const uint32_t *)p)[i]);
    return oracle_half_to_double(((const uint16_t *)p)[i]);
}

/*
 * Step 5: Y[r, j] = sum_k v[r,k] * X[k*b_r + off[r,k], j] in fp64, blocks in
 * ascending order.  X is [N x B] row-major with leading dimension ldx, Y is
 * [M x B] with leading dimension ldy.  B = 1 is the matrix-vector product.
 */
int oracle_spmm_f64(int64_t M, int64_t N, int wdtype, const void *values,
                    const uint8_t *offsets, const uint8_t *log2b, const int64_t *row_start,
                    int xdtype, const void *X, int64_t B, int64_t ldx, double *Y, int64_t ldy) {
    for (int64_t r = 0; r < M; ++r) {
        int64_t b = (int64_t)1 << log2b[r];
        int64_t nblk = (N + b - 1) / b;
        double *y = Y + r * ldy;
        for (int64_t j = 0; j < B; ++j) y[j] = 0.0;
        for (int64_t k = 0; k < nblk; ++k) {
            int64_t s = row_start[r] + k;
            int64_t c = k * b + offsets[s];
            if (offsets[s] >= b || c >= N) return ORACLE_EFORMAT;
            double v = load_elem(wdtype, values, s);
            for (int64_t j = 0; j < B; ++j) y[j] += v * load_elem(xdtype, X, c * ldx + j);
        }
    }
    return ORACLE_OK;
}

/*
 * Same sum, with the magnitudes: A[r, j] = sum_k |v[r,k] * X[c, j]|.  This is the
 * scale a floating-point dot product's rounding error is measured against.
 */
int oracle_spmm_absdot_f64(int64_t M, int64_t N, int wdtype, const void *values,
                           const uint8_t *offsets, const uint8_t *log2b,
                           const int64_t *row_start, int xdtype, const void *X, int64_t B,
                           int64_t ldx, double *A, int64_t lda) {
    for (int64_t r = 0; r < M; ++r) {
        int64_t b = (int64_t)1 << log2b[r];
        int64_t nblk = (N + b - 1) / b;
        double *a = A + r * lda;
        for (int64_t j = 0; j < B; ++j) a[j] = 0.0;
        for (int64_t k = 0; k < nblk; ++k) {
            int64_t s = row_start[r] + k;
            int64_t c = k * b + offsets[s];
            if (offsets[s] >= b || c >= N) return ORACLE_EFORMAT;
            double v = load_elem(wdtype, values, s);
            for (int64_t j = 0; j < B; ++j) a[j] += fabs(v * load_elem(xdtype, X, c * ldx + j));
        }
    }
    return ORACLE_OK;
}

/*
 * Bit-packed offsets (section 4.2: an index inside a block of size b needs only
 * log2 b bits).  Within each block-size group (log2 b = l) the group's slots are
 * numbered j = 0, 1, ... in storage order and cut into runs of 32; run q takes
 * exactly l 32-bit words, and slot j's offset occupies bits (j mod 32) * l ..
 * (j mod 32) * l + l - 1 of the run's l words read as one little-endian bit string.
 * Groups follow each other in storage order; a group of block size 1 takes no
 * words.  first_word[g] receives each group's first word; returns the total words.
 */
int64_t oracle_packed_layout(int64_t M, int64_t N, const uint8_t *log2b, int64_t *first_word) {
    int64_t words = 0;
    for (int l = 0; l <= 7; ++l) {
        int64_t rows = 0;
        for (int64_t r = 0; r < M; ++r) rows += (log2b[r] == l);
        int64_t b = (int64_t)1 << l;
        int64_t slots = rows * ((N + b - 1) / b);
        first_word[l] = words;
        words += (slots + 31) / 32 * l;
    }
    return words;
}

void oracle_pack_offsets(int64_t M, int64_t N, const uint8_t *log2b, const int64_t *row_start,
                         const uint8_t *offsets, uint32_t *packed) {
    int64_t first_word[8];
    int64_t words = oracle_packed_layout(M, N, log2b, first_word);
    for (int64_t w = 0; w < words; ++w) packed[w] = 0u;
    /* the first slot of each group in the grouped storage order */
    int64_t group_first_slot[8];
    for (int l = 0; l <= 7; ++l) group_first_slot[l] = -1;
    for (int64_t r = 0; r < M; ++r) {
        int l = log2b[r];
        if (group_first_slot[l] < 0 || row_start[r] < group_first_slot[l])
            group_first_slot[l] = row_start[r];
    }
    for (int64_t r = 0; r < M; ++r) {
        int l = log2b[r];
        if (l == 0) continue;
        int64_t b = (int64_t)1 << l;
        int64_t nblk = (N + b - 1) / b;
        for (int64_t k = 0; k < nblk; ++k) {
            int64_t j = row_start[r] + k - group_first_slot[l];     /* slot inside its group */
            int64_t bit = (j % 32) * l;
            uint32_t *run = packed + first_word[l] + (j / 32) * l;
            for (int t = 0; t < l; ++t) {                         /* bit by bit, LSB first */
                uint32_t v = (offsets[row_start[r] + k] >> t) & 1u;
                int64_t pos = bit + t;
                run[pos / 32] |= v << (pos % 32);
            }
        }
    }
}

void oracle_unpack_offsets(int64_t M, int64_t N, const uint8_t *log2b, const int64_t *row_start,
                           const uint32_t *packed, uint8_t *offsets) {
    int64_t first_word[8];
    oracle_packed_layout(M, N, log2b, first_word);
    int64_t group_first_slot[8];
    for (int l = 0; l <= 7; ++l) group_first_slot[l] = -1;
    for (int64_t r = 0; r < M; ++r) {
        int l = log2b[r];
        if (group_first_slot[l] < 0 || row_start[r] < group_first_slot[l])
            group_first_slot[l] = row_start[r];
    }
    for (int64_t r = 0; r < M; ++r) {
        int l = log2b[r];
        int64_t b = (int64_t)1 << l;
        int64_t nblk = (N + b - 1) / b;
        for (int64_t k = 0; k < nblk; ++k) {
            uint32_t v = 0;
            if (l > 0) {
                int64_t j = row_start[r] + k - group_first_slot[l];
                int64_t bit = (j % 32) * l;
                const uint32_t *run = packed + first_word[l] + (j / 32) * l;
                for (int t = 0; t < l; ++t) {
                    int64_t pos = bit + t;
                    v |= ((run[pos / 32] >> (pos % 32)) & 1u) << t;
                }
            }
            offsets[row_start[r] + k] = (uint8_t)v;
        }
    }
}

/*
 * Irregular magnitude pruning, the starting point of DARB (section 3.2: the
 * irregular mask is computed only to measure each row's density; section 2
 * describes irregular pruning as keeping the top-K weights by magnitude).
 * Keep the k elements of W with the largest magnitude key (stored bits with the
 * sign cleared, the same key the block-max selection uses); among equal keys the
 * lower flat index r*N + c comes first.  Written as the definition: sort every
 * element by (key descending, flat index ascending), keep the first k, count the
 * kept elements of each row.
 */
typedef struct {
    uint32_t key;
    int64_t idx;
} oracle_ranked;

static int ranked_before(const void *a, const void *b) {
    const oracle_ranked *x = (const oracle_ranked *)a, *y = (const oracle_ranked *)b;
    if (x->key != y->key) return x->key > y->key ? -1 : 1;
    return x->idx < y->idx ? -1 : (x->idx > y->idx ? 1 : 0);
}

int oracle_prune_counts(int64_t M, int64_t N, int dtype, const void *W, int64_t ldw, int64_t k,
                        int64_t *counts) {
    if (M < 1 || N < 1 || ldw < N || k < 0 || k > M * N) return ORACLE_EINVAL;
    if (dtype != DT_F32 && dtype != DT_F16) return ORACLE_EINVAL;
    oracle_ranked *all = (oracle_ranked *)malloc((size_t)(M * N) * sizeof(oracle_ranked));
    if (!all) return ORACLE_EINVAL;
    for (int64_t r = 0; r < M; ++r) {
        for (int64_t c = 0; c < N; ++c) {
            uint32_t key;
            if (dtype == DT_F32) key = ((const uint32_t *)W)[r * ldw + c] & 0x7FFFFFFFu;
            else key = ((const uint16_t *)W)[r * ldw + c] & 0x7FFFu;
            all[r * N + c].key = key;
            all[r * N + c].idx = r * N + c;
        }
    }
    qsort(all, (size_t)(M * N), sizeof(oracle_ranked), ranked_before);
    for (int64_t r = 0; r < M; ++r) counts[r] = 0;
    for (int64_t i = 0; i < k; ++i) counts[all[i].idx / N] += 1;
    free(all);
    return ORACLE_OK;
}
