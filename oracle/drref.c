/*
 * drref.c -- CPU oracle for the DeepReduce sparse-tensor codec
 * (Kostopoulou et al., "DeepReduce: A Sparse-tensor Communication Framework
 * for Distributed Deep Learning", arXiv 2102.03112).
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load this library.  It is a
 * plain, slow, single-threaded statement of what the codec computes, written
 * so that each function can be checked against the paper by eye: no blocking,
 * no fusion, no reordering beyond what the definitions state.  It shares no
 * source, header, table or helper with the GPU library.
 *
 * Readings of the paper that this file fixes where the paper is silent
 * (index base, tie order, rounding of the Bloom parameters, the hash family,
 * the position map, the sort key, the abscissa, the segmentation rule and the
 * width of the reorder map) are stated at the function that applies them.
 *
 * Status codes: 0 ok, -1 invalid argument, -2 output capacity too small
 * (the required count is still reported).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define DRREF_OK 0
#define DRREF_EINVAL (-1)
#define DRREF_ECAPACITY (-2)

/* ------------------------------------------------------------------------ */
/* Hash family.                                                              */
/* ------------------------------------------------------------------------ */

/*
 * The paper asks only for k independent hash functions (Section 2, "Bloom
 * Filter"; Section 4).  This codec uses MurmurHash3_x86_32 (A. Appleby,
 * SMHasher, public domain) with seeds 0..k-1.  The function below is the
 * published algorithm for a byte string of any length; the codec only ever
 * hashes the 4-byte little-endian encoding of a 0-based index.
 */
static uint32_t rotl32(uint32_t x, int r) { return (x << r) | (x >> (32 - r)); }

uint32_t drref_murmur3_32(const uint8_t *data, uint64_t len, uint32_t seed)
{
    const uint32_t c1 = 0xcc9e2d51u;
    const uint32_t c2 = 0x1b873593u;
    uint32_t h = seed;
    uint64_t nblocks = len / 4;
    for (uint64_t b = 0; b < nblocks; ++b) {
        const uint8_t *p = data + 4 * b;
        uint32_t k = (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) |
                     ((uint32_t)p[3] << 24);
        k *= c1;
        k = rotl32(k, 15);
        k *= c2;
        h ^= k;
        h = rotl32(h, 13);
        h = h * 5u + 0xe6546b64u;
    }
    const uint8_t *tail = data + 4 * nblocks;
    uint32_t k = 0;
    switch (len & 3) {
    case 3:
        k ^= (uint32_t)tail[2] << 16; /* fall through */
    case 2:
        k ^= (uint32_t)tail[1] << 8; /* fall through */
    case 1:
        k ^= (uint32_t)tail[0];
        k *= c1;
        k = rotl32(k, 15);
        k *= c2;
        h ^= k;
    }
    h ^= (uint32_t)len;
    /* final avalanche */
    h ^= h >> 16;
    h *= 0x85ebca6bu;
    h ^= h >> 13;
    h *= 0xc2b2ae35u;
    h ^= h >> 16;
    return h;
}

/*
 * Bit position of hash function j for index i in an m-bit filter.
 * h_j(i) is the hash of the 4-byte little-endian encoding of i with seed j.
 * It is mapped to [0, m) by floor(h * m / 2^32) (Lemire's multiply-shift
 * range reduction), which needs m < 2^32.
 */
uint64_t drref_bloom_pos(uint32_t i, uint32_t j, uint64_t m)
{
    uint8_t le[4] = {(uint8_t)(i & 0xff), (uint8_t)((i >> 8) & 0xff), (uint8_t)((i >> 16) & 0xff),
                     (uint8_t)((i >> 24) & 0xff)};
    uint32_t h = drref_murmur3_32(le, 4, j);
    return ((uint64_t)h * m) >> 32;
}

void drref_bloom_pos_many(const uint32_t *idx, uint64_t n, uint32_t j, uint64_t m, uint64_t *out)
{
    for (uint64_t q = 0; q < n; ++q)
        out[q] = drref_bloom_pos(idx[q], j, m);
}

/*
 * Filter layouts.  STANDARD (0): every hash function addresses the whole
 * m-bit array, as above.  PARTITIONED (1): the array is cut into k parts,
 * part j covering bits [floor(j m / k), floor((j+1) m / k)), and hash
 * function j addresses only part j: pos_j(i) = floor(j m / k) +
 * floor(h_j(i) q_j / 2^32) with q_j the part's size.  Section 2 asks only for
 * k independent hash functions into the m-bit array; in the partitioned
 * array each part receives n insertions into about m/k bits, so a part's
 * fill is about 1 - e^{-kn/m} and the false-positive rate about
 * (1 - e^{-kn/m})^k, the same as Lemma 2 gives for the standard array.
 * The same Murmur hash and seeds are used.  (The partitioned layout is the
 * one a GPU can query with its first parts held in on-chip memory.)
 */
#define DRREF_LAYOUT_STANDARD 0u
#define DRREF_LAYOUT_PARTITIONED 1u

uint64_t drref_part_start(uint32_t j, uint64_t m, uint32_t k) { return (uint64_t)j * m / k; }

uint64_t drref_bloom_pos_layout(uint32_t i, uint32_t j, uint64_t m, uint32_t k, uint32_t layout)
{
    if (layout == DRREF_LAYOUT_STANDARD)
        return drref_bloom_pos(i, j, m);
    uint64_t lo = drref_part_start(j, m, k), hi = drref_part_start(j + 1, m, k);
    uint8_t le[4] = {(uint8_t)(i & 0xff), (uint8_t)((i >> 8) & 0xff), (uint8_t)((i >> 16) & 0xff),
                     (uint8_t)((i >> 24) & 0xff)};
    uint32_t h = drref_murmur3_32(le, 4, j);
    return lo + (((uint64_t)h * (hi - lo)) >> 32);
}

void drref_bloom_pos_layout_many(const uint32_t *idx, uint64_t n, uint32_t j, uint64_t m, uint32_t k, uint32_t layout,
                                 uint64_t *out)
{
    for (uint64_t q = 0; q < n; ++q)
        out[q] = drref_bloom_pos_layout(idx[q], j, m, k, layout);
}

/* ------------------------------------------------------------------------ */
/* Bloom filter parameters (Lemma 2 and Remark 2, Section 10.2).             */
/* ------------------------------------------------------------------------ */

/*
 * Remark 2 gives the optimal real-valued size m = -n ln(eps) / (ln 2)^2 and
 * hash count k = -ln(eps) / ln 2.  Integer reading used here:
 *   k = max(1, round-half-away(-ln(eps) / ln 2))
 *   C = -ln(eps) / (ln 2 * ln 2);  m = 32 * ceil(ceil(n * C) / 32), at least 32.
 * Everything is IEEE double with the C library's log.
 */
int drref_bloom_params(uint64_t n, double fpr, uint64_t *m_out, uint32_t *k_out)
{
    if (!(fpr > 0.0 && fpr < 1.0) || !m_out || !k_out)
        return DRREF_EINVAL;
    double ln2 = log(2.0);
    double kk = -log(fpr) / ln2;
    long kr = lround(kk);
    if (kr < 1)
        kr = 1;
    double C = -log(fpr) / (ln2 * ln2);
    double raw = ceil((double)n * C);
    uint64_t m = (uint64_t)raw;
    m = ((m + 31) / 32) * 32;
    if (m < 32)
        m = 32;
    if (m >= ((uint64_t)1 << 32))
        return DRREF_EINVAL;
    *m_out = m;
    *k_out = (uint32_t)kr;
    return DRREF_OK;
}

/* ------------------------------------------------------------------------ */
/* Top-r sparsification (Section 2 "Sparsification"; Section 10.2).         */
/* ------------------------------------------------------------------------ */

/* Magnitude key: the IEEE bit pattern with the sign cleared.  For non-NaN
 * floats it orders exactly like |x|, and +0 and -0 both map to 0. */
static uint32_t mag_key(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    return u & 0x7fffffffu;
}

typedef struct {
    uint32_t key;
    uint32_t idx;
} key_idx;

/* key descending, then index ascending: a strict total order */
static int cmp_key_desc_idx_asc(const void *a, const void *b)
{
    const key_idx *x = (const key_idx *)a, *y = (const key_idx *)b;
    if (x->key != y->key)
        return x->key > y->key ? -1 : 1;
    if (x->idx != y->idx)
        return x->idx < y->idx ? -1 : 1;
    return 0;
}

static int cmp_u32_asc(const void *a, const void *b)
{
    uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
    return (x > y) - (x < y);
}

static int has_nonfinite(const float *g, uint64_t d)
{
    for (uint64_t i = 0; i < d; ++i)
        if (!isfinite(g[i]))
            return 1;
    return 0;
}

/*
 * Top-r: S holds the indices of the r entries of largest magnitude.  Ties in
 * magnitude are broken by smaller index first (the paper does not say).  S is
 * returned in ascending index order, which is the order the receiver's loop
 * over [d] visits them (Section 4).  Indices are 0-based.
 * Non-finite input is rejected.
 */
int drref_topr(const float *g, uint64_t d, uint64_t r, uint32_t *S_out)
{
    if ((!g && d) || (!S_out && r) || r > d || d >= ((uint64_t)1 << 32))
        return DRREF_EINVAL;
    if (has_nonfinite(g, d))
        return DRREF_EINVAL;
    if (r == 0)
        return DRREF_OK;
    key_idx *a = (key_idx *)malloc(sizeof(key_idx) * d);
    if (!a)
        return DRREF_EINVAL;
    for (uint64_t i = 0; i < d; ++i) {
        a[i].key = mag_key(g[i]);
        a[i].idx = (uint32_t)i;
    }
    qsort(a, d, sizeof(key_idx), cmp_key_desc_idx_asc);
    for (uint64_t q = 0; q < r; ++q)
        S_out[q] = a[q].idx;
    free(a);
    qsort(S_out, r, sizeof(uint32_t), cmp_u32_asc);
    return DRREF_OK;
}

/*
 * Inherently sparse input (Section 3; the NCF experiment of Section 6.3):
 * S is the support {i : g[i] != 0}, ascending.  -0.0 counts as zero.
 */
int drref_nonzero(const float *g, uint64_t d, uint32_t *S_out, uint64_t cap, uint64_t *n_out)
{
    if ((!g && d) || !n_out || d >= ((uint64_t)1 << 32))
        return DRREF_EINVAL;
    if (has_nonfinite(g, d))
        return DRREF_EINVAL;
    uint64_t n = 0;
    for (uint64_t i = 0; i < d; ++i) {
        if (g[i] != 0.0f) {
            if (n < cap)
                S_out[n] = (uint32_t)i;
            ++n;
        }
    }
    *n_out = n;
    return n > cap ? DRREF_ECAPACITY : DRREF_OK;
}

/* ------------------------------------------------------------------------ */
/* Bloom filter insert and full-range query (Sections 2 and 4).              */
/* ------------------------------------------------------------------------ */

/* Bit p of the filter lives in 32-bit word p/32 at bit p%32 (LSB first). */
static int get_bit(const uint32_t *w, uint64_t p) { return (int)((w[p >> 5] >> (p & 31)) & 1u); }
static void set_bit(uint32_t *w, uint64_t p) { w[p >> 5] |= 1u << (p & 31); }

/* Insert every s in S: set bit h_j(s) for j = 0..k-1 (Section 2), in the
 * given layout. */
int drref_bloom_encode_layout(const uint32_t *S, uint64_t n, uint64_t m, uint32_t k, uint32_t layout,
                              uint32_t *words)
{
    if ((!S && n) || !words || m < 32 || (m & 31) || m >= ((uint64_t)1 << 32) || k < 1 || k > 32 ||
        layout > DRREF_LAYOUT_PARTITIONED)
        return DRREF_EINVAL;
    memset(words, 0, sizeof(uint32_t) * (m / 32));
    for (uint64_t q = 0; q < n; ++q)
        for (uint32_t j = 0; j < k; ++j)
            set_bit(words, drref_bloom_pos_layout(S[q], j, m, k, layout));
    return DRREF_OK;
}

int drref_bloom_encode(const uint32_t *S, uint64_t n, uint64_t m, uint32_t k, uint32_t *words)
{
    return drref_bloom_encode_layout(S, n, m, k, DRREF_LAYOUT_STANDARD, words);
}

/* Membership: i is reported iff all k of its bits are set (Section 4,
 * "Implementation on GPUs and CPUs": the k looked-up bits sum to k). */
static int bloom_member(const uint32_t *words, uint64_t m, uint32_t k, uint32_t layout, uint32_t i)
{
    for (uint32_t j = 0; j < k; ++j)
        if (!get_bit(words, drref_bloom_pos_layout(i, j, m, k, layout)))
            return 0;
    return 1;
}

/*
 * Full-range query, policy P0 (Section 4, "No-error approach"): visit every
 * i of the gradient's index range in increasing order and collect the
 * positives, true and false, into P.  P is therefore ascending.
 */
int drref_bloom_query_layout(const uint32_t *words, uint64_t m, uint32_t k, uint32_t layout, uint64_t d,
                             uint32_t *P_out, uint64_t cap, uint64_t *n_out)
{
    if (!words || !n_out || m < 32 || (m & 31) || m >= ((uint64_t)1 << 32) || k < 1 || k > 32 ||
        d >= ((uint64_t)1 << 32) || layout > DRREF_LAYOUT_PARTITIONED)
        return DRREF_EINVAL;
    uint64_t n = 0;
    for (uint64_t i = 0; i < d; ++i) {
        if (bloom_member(words, m, k, layout, (uint32_t)i)) {
            if (n < cap)
                P_out[n] = (uint32_t)i;
            ++n;
        }
    }
    *n_out = n;
    return n > cap ? DRREF_ECAPACITY : DRREF_OK;
}

int drref_bloom_query(const uint32_t *words, uint64_t m, uint32_t k, uint64_t d, uint32_t *P_out,
                      uint64_t cap, uint64_t *n_out)
{
    return drref_bloom_query_layout(words, m, k, DRREF_LAYOUT_STANDARD, d, P_out, cap, n_out);
}

/* ------------------------------------------------------------------------ */
/* Curve fitting of the values (Section 5; Section 5.1 for the reorder map). */
/* ------------------------------------------------------------------------ */

/* Order-preserving map of a float to u32 (unsigned order == float order,
 * with -0 just below +0). */
static uint32_t order_key(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

/*
 * Descending sort of the values (Section 5: the nonzero values are sorted in
 * descending order).  Signed order; equal values keep their original order.
 * perm_out[rank] = original position q of the value with that rank.
 */
int drref_sort_desc(const float *V, uint64_t n, uint32_t *perm_out)
{
    if ((!V || !perm_out) && n)
        return DRREF_EINVAL;
    if (n == 0)
        return DRREF_OK;
    key_idx *a = (key_idx *)malloc(sizeof(key_idx) * n);
    if (!a)
        return DRREF_EINVAL;
    for (uint64_t q = 0; q < n; ++q) {
        a[q].key = order_key(V[q]);
        a[q].idx = (uint32_t)q;
    }
    qsort(a, n, sizeof(key_idx), cmp_key_desc_idx_asc); /* order key descending, q ascending */
    for (uint64_t q = 0; q < n; ++q)
        perm_out[q] = a[q].idx;
    free(a);
    return DRREF_OK;
}

/*
 * Least-squares polynomial of degree D through the points (x_j, y_j)
 * (Section 5, "Polynomial regression"): minimise sum_j (y_j - sum_p c_p x_j^p)^2.
 * Normal equations G c = b with G[p][q] = sum_j x_j^(p+q), b[p] = sum_j x_j^p y_j,
 * accumulated in double in increasing j, solved by Gaussian elimination with
 * partial pivoting.  coef_out[p] multiplies x^p.
 */
#define DRREF_MAX_DEG 7
int drref_lsq_fit(const double *x, const double *y, uint64_t n, uint32_t D, double *coef_out)
{
    if (D > DRREF_MAX_DEG || n < (uint64_t)D + 1 || !x || !y || !coef_out)
        return DRREF_EINVAL;
    const int N = (int)D + 1;
    double powsum[2 * DRREF_MAX_DEG + 1];
    double rhs[DRREF_MAX_DEG + 1];
    for (int e = 0; e <= 2 * (int)D; ++e)
        powsum[e] = 0.0;
    for (int p = 0; p < N; ++p)
        rhs[p] = 0.0;
    for (uint64_t j = 0; j < n; ++j) {
        double tp = 1.0;
        for (int e = 0; e <= 2 * (int)D; ++e) {
            powsum[e] += tp;
            if (e < N)
                rhs[e] += tp * y[j];
            tp *= x[j];
        }
    }
    double A[DRREF_MAX_DEG + 1][DRREF_MAX_DEG + 2];
    for (int p = 0; p < N; ++p) {
        for (int q = 0; q < N; ++q)
            A[p][q] = powsum[p + q];
        A[p][N] = rhs[p];
    }
    for (int col = 0; col < N; ++col) {
        int piv = col;
        for (int row = col + 1; row < N; ++row)
            if (fabs(A[row][col]) > fabs(A[piv][col]))
                piv = row;
        if (A[piv][col] == 0.0)
            return DRREF_EINVAL;
        if (piv != col)
            for (int c = 0; c <= N; ++c) {
                double t = A[col][c];
                A[col][c] = A[piv][c];
                A[piv][c] = t;
            }
        for (int row = col + 1; row < N; ++row) {
            double f = A[row][col] / A[col][col];
            for (int c = col; c <= N; ++c)
                A[row][c] -= f * A[col][c];
        }
    }
    for (int p = N - 1; p >= 0; --p) {
        double s = A[p][N];
        for (int q = p + 1; q < N; ++q)
            s -= A[p][q] * coef_out[q];
        coef_out[p] = s / A[p][p];
    }
    return DRREF_OK;
}

/*
 * Segmentation and degree actually used for n sorted values, requested
 * degree D and requested segment count S.  Segments hold equal counts of
 * consecutive sorted values; a segment is never given fewer than D+1 points
 * (Section 5 stops splitting below n'+1 points):
 *   S_eff = min(S, max(1, floor(n / (D+1)))),
 *   D_eff = D if n >= D+1, else n-1 (interpolation through all points).
 * Segment s covers ranks [floor(s n / S_eff), floor((s+1) n / S_eff)).
 */
void drref_fit_shape(uint64_t n, uint32_t D, uint32_t S, uint32_t *S_eff, uint32_t *D_eff)
{
    if (n == 0) {
        *S_eff = 0;
        *D_eff = 0;
        return;
    }
    uint64_t cap = n / ((uint64_t)D + 1);
    if (cap < 1)
        cap = 1;
    *S_eff = (uint32_t)((uint64_t)S < cap ? (uint64_t)S : cap);
    *D_eff = n >= (uint64_t)D + 1 ? D : (uint32_t)(n - 1);
}

static uint64_t seg_lo(uint64_t s, uint64_t n, uint64_t S_eff) { return s * n / S_eff; }

/*
 * Abscissa of local rank j in a segment of n_s points.  The paper fits the
 * points (i, C_S(g)[i]) with i the rank (Section 5).  The same least-squares
 * problem is posed here in the affine image t = (2j - (n_s - 1)) / (n_s - 1)
 * of the rank, which maps the segment onto [-1, 1] and keeps the normal
 * equations well conditioned; the fitted curve is the same function of the
 * rank.  t = 0 for a one-point segment.
 */
static double abscissa(uint64_t j, uint64_t n_s)
{
    if (n_s <= 1)
        return 0.0;
    return (double)(2 * (int64_t)j - (int64_t)(n_s - 1)) / (double)(n_s - 1);
}

/* Width of one reorder-map entry (Section 5.1): the smallest b >= 1 with
 * 2^b >= n, i.e. ceil(log2 n) bits per value. */
uint32_t drref_sigma_bits(uint64_t n)
{
    uint32_t b = 1;
    while (b < 63 && ((uint64_t)1 << b) < n)
        ++b;
    return b;
}

uint64_t drref_sigma_words(uint64_t n)
{
    return (n * drref_sigma_bits(n) + 31) / 32;
}

/* ------------------------------------------------------------------------ */
/* Double-exponential value fit (Section 5, "Nonlinear regression").        */
/* ------------------------------------------------------------------------ */

#define DRREF_DEXP_ITERS 40
#define DRREF_DEXP_RATE_MAX 40.0

/* Solve the n x n system A x = rhs (n <= 4) by Gaussian elimination with
 * partial pivoting; nonzero if a pivot is zero. */
static int solve_small(int n, double A[4][5], double *x)
{
    for (int col = 0; col < n; ++col) {
        int piv = col;
        for (int row = col + 1; row < n; ++row)
            if (fabs(A[row][col]) > fabs(A[piv][col]))
                piv = row;
        if (A[piv][col] == 0.0)
            return 1;
        if (piv != col)
            for (int c = 0; c <= n; ++c) {
                double t = A[col][c];
                A[col][c] = A[piv][c];
                A[piv][c] = t;
            }
        for (int row = col + 1; row < n; ++row) {
            double f = A[row][col] / A[col][col];
            for (int c = col; c <= n; ++c)
                A[row][c] -= f * A[col][c];
        }
    }
    for (int p = n - 1; p >= 0; --p) {
        double s = A[p][n];
        for (int q = p + 1; q < n; ++q)
            s -= A[p][q] * x[q];
        x[p] = s / A[p][p];
    }
    return 0;
}

/*
 * Sums of one pass over the points for y ~ a e^(b t) + c e^(d t): the upper
 * triangle of J^T J (row-major: 00 01 02 03 11 12 13 22 23 33), J^T r and
 * r^T r, with J = [e^(bt), a t e^(bt), e^(dt), c t e^(dt)] and r = y - model,
 * accumulated in double in increasing j.
 */
static void dexp_sums(const double *t, const double *y, uint64_t n, const double th[4], double s[15])
{
    for (int e = 0; e < 15; ++e)
        s[e] = 0.0;
    for (uint64_t j = 0; j < n; ++j) {
        const double eb = exp(th[1] * t[j]), ed = exp(th[3] * t[j]);
        const double J[4] = {eb, th[0] * t[j] * eb, ed, th[2] * t[j] * ed};
        const double r = y[j] - (th[0] * eb + th[2] * ed);
        int e = 0;
        for (int p = 0; p < 4; ++p)
            for (int q = p; q < 4; ++q)
                s[e++] += J[p] * J[q];
        for (int p = 0; p < 4; ++p)
            s[10 + p] += J[p] * r;
        s[14] += r * r;
    }
}

/*
 * Least-squares fit of y_j ~ a e^(b t_j) + c e^(d t_j) over n >= 4 points
 * (Section 5 names the model; its fitting method is not given).  Steps:
 *  1. start from rates b = 1, d = -1 and the amplitudes (a, c) that solve
 *     the 2 x 2 linear least-squares problem for those rates (a = mean y,
 *     c = 0 if it is singular);
 *  2. DRREF_DEXP_ITERS Levenberg-Marquardt steps: solve
 *     (J^T J + lambda diag(J^T J)) delta = J^T r, clamp the rates of
 *     theta + delta to [-40, 40], and keep the trial point if its residual
 *     sum of squares is smaller (lambda /= 10), else keep theta (lambda *=
 *     10); lambda starts at 1e-3 and a singular system counts as a reject.
 * theta_out = (a, b, c, d); *rss_out = the final residual sum of squares.
 */
int drref_dexp_fit(const double *t, const double *y, uint64_t n, double *theta_out, double *rss_out)
{
    if (!t || !y || !theta_out || n < 4)
        return DRREF_EINVAL;
    double th[4] = {0.0, 1.0, 0.0, -1.0};
    {
        double s11 = 0, s12 = 0, s22 = 0, sy1 = 0, sy2 = 0, sy = 0;
        for (uint64_t j = 0; j < n; ++j) {
            const double e1 = exp(t[j]), e2 = exp(-t[j]);
            s11 += e1 * e1;
            s12 += e1 * e2;
            s22 += e2 * e2;
            sy1 += y[j] * e1;
            sy2 += y[j] * e2;
            sy += y[j];
        }
        const double det = s11 * s22 - s12 * s12;
        if (det != 0.0) {
            th[0] = (sy1 * s22 - sy2 * s12) / det;
            th[2] = (sy2 * s11 - sy1 * s12) / det;
        } else {
            th[0] = sy / (double)n;
        }
    }
    double s[15], st[15];
    dexp_sums(t, y, n, th, s);
    double lambda = 1e-3;
    for (int it = 0; it < DRREF_DEXP_ITERS; ++it) {
        double A[4][5];
        int e = 0;
        for (int p = 0; p < 4; ++p)
            for (int q = p; q < 4; ++q) {
                A[p][q] = s[e];
                A[q][p] = s[e];
                ++e;
            }
        for (int p = 0; p < 4; ++p) {
            A[p][p] += lambda * A[p][p];
            A[p][4] = s[10 + p];
        }
        double delta[4];
        if (solve_small(4, A, delta)) {
            lambda *= 10.0;
            continue;
        }
        double tt[4];
        for (int p = 0; p < 4; ++p)
            tt[p] = th[p] + delta[p];
        for (int p = 1; p < 4; p += 2)
            tt[p] = tt[p] > DRREF_DEXP_RATE_MAX ? DRREF_DEXP_RATE_MAX
                                                : (tt[p] < -DRREF_DEXP_RATE_MAX ? -DRREF_DEXP_RATE_MAX : tt[p]);
        dexp_sums(t, y, n, tt, st);
        if (st[14] < s[14]) {
            for (int p = 0; p < 4; ++p)
                th[p] = tt[p];
            for (int q = 0; q < 15; ++q)
                s[q] = st[q];
            lambda /= 10.0;
        } else {
            lambda *= 10.0;
        }
    }
    for (int p = 0; p < 4; ++p)
        theta_out[p] = th[p];
    if (rss_out)
        *rss_out = s[14];
    return DRREF_OK;
}

/* ------------------------------------------------------------------------ */
/* Adaptive segmentation (Section 5, "Piece-wise approximation") and the    */
/* number of pieces (Section 5 after Lemma 1; Remark 4 of Section 10).     */
/* ------------------------------------------------------------------------ */

#define DRREF_MAX_SEG 4096
#define DRREF_SEG_EQUAL 0u
#define DRREF_SEG_CHORD 1u

/*
 * Distance of sorted value C[i] from the chord through the segment's first
 * and last points (ranks a and z > a).  The paper takes the squared vertical
 * distance; its absolute value has the same maximiser.  Evaluated in double
 * as written, one rounding per operation (no fused multiply-add), so that
 * any implementation that follows these steps takes the same decisions.
 */
static double chord_dist(const float *C, uint64_t a, uint64_t z, uint64_t i)
{
    const double ca = (double)C[a];
    const double m = ((double)C[z] - ca) / (double)(z - a);
    const double y = ca + m * (double)(i - a);
    return fabs(y - (double)C[i]);
}

/*
 * Farthest allowed split point of segment [a, e) for degree D: the rank i
 * that ends the left part, over the ranks that leave both parts at least
 * D+1 points (the paper stops below n'+1 points); ties to the smaller rank.
 * Returns 0 and leaves *i_out alone if no split is allowed.
 */
static double seg_candidate(const float *C, uint64_t a, uint64_t e, uint32_t D, uint64_t *i_out)
{
    const uint64_t minpts = (uint64_t)D + 1;
    if (e - a < 2 * minpts)
        return 0.0;
    const uint64_t z = e - 1;
    double best = 0.0;
    for (uint64_t i = a + D; i + minpts <= z; ++i) {
        const double dd = chord_dist(C, a, z, i);
        if (dd > best) {
            best = dd;
            *i_out = i;
        }
    }
    return best;
}

/*
 * Segment starts of the sorted values C[0..n) (descending), for degree D and
 * at most S segments: bounds_out[0..S_eff] with bounds_out[0] = 0 and
 * bounds_out[S_eff] = n.
 *  - Equal-count segments: segment s covers [floor(s n / S_eff),
 *    floor((s+1) n / S_eff)), S_eff as in drref_fit_shape.
 *  - Chord segmentation (Section 5): the values with the sign bit clear and
 *    the rest (positive and negative sorted values) start as separate
 *    segments, when S >= 2 and both hold at least D+1 points.  Then, while
 *    there are fewer than S segments, the segment whose farthest allowed
 *    split point lies farthest from its chord (ties: the leftmost segment)
 *    is split after that point.  It stops early when no segment has an
 *    allowed split point off its chord.
 */
int drref_segment(const float *C, uint64_t n, uint32_t D, uint32_t S, uint32_t mode, uint64_t *bounds_out,
                  uint32_t *S_eff_out)
{
    if ((!C && n) || !bounds_out || !S_eff_out || S < 1 || S > DRREF_MAX_SEG || mode > DRREF_SEG_CHORD ||
        D > DRREF_MAX_DEG)
        return DRREF_EINVAL;
    bounds_out[0] = 0;
    if (n == 0) {
        *S_eff_out = 0;
        return DRREF_OK;
    }
    if (mode == DRREF_SEG_EQUAL) {
        uint32_t S_eff, D_eff;
        drref_fit_shape(n, D, S, &S_eff, &D_eff);
        for (uint32_t s = 0; s <= S_eff; ++s)
            bounds_out[s] = (uint64_t)s * n / S_eff;
        *S_eff_out = S_eff;
        return DRREF_OK;
    }
    const uint64_t minpts = (uint64_t)D + 1;
    uint64_t l = 0;
    while (l < n && !signbit(C[l]))
        ++l;
    uint32_t count = 1;
    bounds_out[1] = n;
    if (S >= 2 && l >= minpts && n - l >= minpts) {
        bounds_out[1] = l;
        bounds_out[2] = n;
        count = 2;
    }
    while (count < S) {
        int64_t best_seg = -1;
        double best = 0.0;
        uint64_t best_i = 0;
        for (uint32_t k = 0; k < count; ++k) {
            uint64_t i = 0;
            const double dd = seg_candidate(C, bounds_out[k], bounds_out[k + 1], D, &i);
            if (dd > best) {
                best = dd;
                best_seg = k;
                best_i = i;
            }
        }
        if (best_seg < 0)
            break;
        for (uint32_t k = count + 1; k > (uint32_t)best_seg + 1; --k)
            bounds_out[k] = bounds_out[k - 1];
        bounds_out[best_seg + 1] = best_i + 1;
        ++count;
    }
    *S_eff_out = count;
    return DRREF_OK;
}

/*
 * Number of segments when the caller asks for the heuristic: p + 1 pieces
 * for p knots, with M = |(C[0] - C[1]) - (C[n-2] - C[n-1])| (the first and
 * last differences of the sorted curve; 0 if n < 2), and
 *  - p = ceil(2 sqrt(M)) for a fit of degree >= 1 (Section 5, from the
 *    piece-wise linear bound 2M/p^2 of Lemma 1),
 *  - p = ceil(M / sqrt(2) - 1) for degree 0 (Remark 4, piece-wise constant),
 * at least 0, and at most DRREF_MAX_SEG pieces.  Each ceiling is found as the
 * smallest p >= 0 with p^2 >= 4M, resp. 2 (p+1)^2 >= M^2, in double, which
 * needs no square root.
 */
uint32_t drref_seg_heuristic(const float *C, uint64_t n, uint32_t D)
{
    double M = 0.0;
    if (n >= 2)
        M = fabs(((double)C[0] - (double)C[1]) - ((double)C[n - 2] - (double)C[n - 1]));
    uint32_t p = 0;
    if (D == 0) {
        const double M2 = M * M;
        while (p + 1 < DRREF_MAX_SEG && 2.0 * (double)(p + 1) * (double)(p + 1) < M2)
            ++p;
    } else {
        const double M4 = 4.0 * M;
        while (p + 1 < DRREF_MAX_SEG && (double)p * (double)p < M4)
            ++p;
    }
    return p + 1;
}

/*
 * Value encoder (Section 5 and 5.1).  Sort V descending; split the sorted
 * curve into equal-count segments; fit each by least squares in double;
 * store the coefficients as fp32, S_eff rows of stride D+1 with unused
 * entries zero.  The reorder map sigma[q] = rank of V[q] in the sorted order
 * (original position -> final position) is packed LSB-first, b bits per
 * entry, entry q in bits [q b, (q+1) b) of the word stream.
 * coef64_out (optional) receives the double-precision coefficients.
 */
/*
 * The same with a choice of segmentation: mode DRREF_SEG_EQUAL or
 * DRREF_SEG_CHORD (drref_segment), and S = 0 for the heuristic number of
 * segments (drref_seg_heuristic).  coef_out and coef64_out hold
 * S_cap = (S ? S : DRREF_MAX_SEG) rows; bounds_out (optional) S_cap + 1
 * segment starts.
 */
#define DRREF_FIT_POLY 0u
#define DRREF_FIT_DEXP 1u

static int curvefit_encode_impl(const float *V, uint64_t n, uint32_t D, uint32_t S, uint32_t mode, uint32_t model,
                                float *coef_out, double *coef64_out, uint32_t *sigma_out, uint64_t *bounds_out,
                                uint32_t *S_eff_out, uint32_t *D_eff_out, uint32_t *b_out);

/*
 * The general value encoder: model DRREF_FIT_POLY (polynomials of degree D)
 * or DRREF_FIT_DEXP (a e^(bt) + c e^(dt) per run, coefficient row (a, b, c,
 * d); D is taken as 3, the four parameters needing at least four points per
 * run).  A DEXP tensor of fewer than four values is coded as the polynomial
 * through them; *model_out reports the model used.
 */
int drref_curvefit_encode_ex(const float *V, uint64_t n, uint32_t D, uint32_t S, uint32_t mode, uint32_t model,
                             float *coef_out, double *coef64_out, uint32_t *sigma_out, uint64_t *bounds_out,
                             uint32_t *S_eff_out, uint32_t *D_eff_out, uint32_t *b_out, uint32_t *model_out)
{
    if (model > DRREF_FIT_DEXP || !model_out)
        return DRREF_EINVAL;
    if (model == DRREF_FIT_DEXP)
        D = 3;
    *model_out = (model == DRREF_FIT_DEXP && n >= 4) ? DRREF_FIT_DEXP : DRREF_FIT_POLY;
    return curvefit_encode_impl(V, n, D, S, mode, *model_out, coef_out, coef64_out, sigma_out, bounds_out,
                                S_eff_out, D_eff_out, b_out);
}

int drref_curvefit_encode_seg(const float *V, uint64_t n, uint32_t D, uint32_t S, uint32_t mode,
                              float *coef_out, double *coef64_out, uint32_t *sigma_out, uint64_t *bounds_out,
                              uint32_t *S_eff_out, uint32_t *D_eff_out, uint32_t *b_out)
{
    return curvefit_encode_impl(V, n, D, S, mode, DRREF_FIT_POLY, coef_out, coef64_out, sigma_out, bounds_out,
                                S_eff_out, D_eff_out, b_out);
}

static int curvefit_encode_impl(const float *V, uint64_t n, uint32_t D, uint32_t S, uint32_t mode, uint32_t model,
                                float *coef_out, double *coef64_out, uint32_t *sigma_out, uint64_t *bounds_out,
                                uint32_t *S_eff_out, uint32_t *D_eff_out, uint32_t *b_out)
{
    if ((!V && n) || D > DRREF_MAX_DEG || S > DRREF_MAX_SEG || mode > DRREF_SEG_CHORD || !coef_out ||
        (!sigma_out && n) || !S_eff_out || !D_eff_out || !b_out)
        return DRREF_EINVAL;
    for (uint64_t q = 0; q < n; ++q)
        if (!isfinite(V[q]))
            return DRREF_EINVAL;
    const uint32_t S_cap = S ? S : DRREF_MAX_SEG;
    uint32_t S_unused, D_eff;
    drref_fit_shape(n, D, S_cap, &S_unused, &D_eff);
    *D_eff_out = D_eff;
    *b_out = drref_sigma_bits(n);
    for (uint64_t c = 0; c < (uint64_t)S_cap * (D + 1); ++c) {
        coef_out[c] = 0.0f;
        if (coef64_out)
            coef64_out[c] = 0.0;
    }
    if (n == 0) {
        *S_eff_out = 0;
        if (bounds_out)
            bounds_out[0] = 0;
        return DRREF_OK;
    }

    uint32_t *perm = (uint32_t *)malloc(sizeof(uint32_t) * n);
    double *xs = (double *)malloc(sizeof(double) * n);
    double *ys = (double *)malloc(sizeof(double) * n);
    float *C = (float *)malloc(sizeof(float) * n);
    uint64_t *bounds = (uint64_t *)malloc(sizeof(uint64_t) * ((size_t)S_cap + 1));
    if (!perm || !xs || !ys || !C || !bounds) {
        free(perm);
        free(xs);
        free(ys);
        free(C);
        free(bounds);
        return DRREF_EINVAL;
    }
    int st = drref_sort_desc(V, n, perm);
    uint32_t S_eff = 0;
    if (st == DRREF_OK) {
        for (uint64_t j = 0; j < n; ++j)
            C[j] = V[perm[j]];
        const uint32_t S_req = S ? S : drref_seg_heuristic(C, n, D);
        st = drref_segment(C, n, D, S_req, mode, bounds, &S_eff);
    }
    *S_eff_out = S_eff;
    if (bounds_out && st == DRREF_OK)
        for (uint32_t s = 0; s <= S_eff; ++s)
            bounds_out[s] = bounds[s];
    for (uint32_t s = 0; st == DRREF_OK && s < S_eff; ++s) {
        uint64_t lo = bounds[s], hi = bounds[s + 1];
        uint64_t ns = hi - lo;
        for (uint64_t j = 0; j < ns; ++j) {
            xs[j] = abscissa(j, ns);
            ys[j] = (double)V[perm[lo + j]];
        }
        double c[DRREF_MAX_DEG + 1];
        /* a chord segment holds at least D+1 points; one of an equal-count
         * split too, unless n < D+1, when D_eff = n-1 interpolates */
        if (model == DRREF_FIT_DEXP)
            st = drref_dexp_fit(xs, ys, ns, c, NULL);
        else
            st = drref_lsq_fit(xs, ys, ns, D_eff, c);
        for (uint32_t p = 0; st == DRREF_OK && p <= D_eff; ++p) {
            coef_out[(uint64_t)s * (D + 1) + p] = (float)c[p];
            if (coef64_out)
                coef64_out[(uint64_t)s * (D + 1) + p] = c[p];
        }
    }
    if (st == DRREF_OK) {
        uint32_t b = *b_out;
        uint64_t nw = (n * b + 31) / 32;
        memset(sigma_out, 0, sizeof(uint32_t) * nw);
        for (uint64_t rank = 0; rank < n; ++rank) {
            uint64_t q = perm[rank];
            /* write value `rank` into bits [q b, (q+1) b) */
            for (uint32_t t = 0; t < b; ++t)
                if ((rank >> t) & 1u)
                    set_bit(sigma_out, q * b + t);
        }
    }
    free(perm);
    free(xs);
    free(ys);
    free(C);
    free(bounds);
    return st;
}

int drref_curvefit_encode(const float *V, uint64_t n, uint32_t D, uint32_t S, float *coef_out,
                          double *coef64_out, uint32_t *sigma_out, uint32_t *S_eff_out,
                          uint32_t *D_eff_out, uint32_t *b_out)
{
    if (S < 1)
        return DRREF_EINVAL;
    return drref_curvefit_encode_seg(V, n, D, S, DRREF_SEG_EQUAL, coef_out, coef64_out, sigma_out, NULL,
                                     S_eff_out, D_eff_out, b_out);
}

/* Read entry q of a packed b-bit stream. */
static uint64_t sigma_get(const uint32_t *sigma, uint64_t q, uint32_t b)
{
    uint64_t v = 0;
    for (uint32_t t = 0; t < b; ++t)
        v |= (uint64_t)get_bit(sigma, q * b + t) << t;
    return v;
}

/*
 * Value decoder.  For each position q: read its rank from sigma, find the
 * segment holding that rank and the rank's local index, and evaluate that
 * segment's polynomial at the abscissa by Horner's rule in double on the
 * fp32 coefficients; round to fp32.  A rank outside [0, n) is an invalid
 * payload.
 */
int drref_curvefit_decode_ex(const float *coef, const uint32_t *sigma, uint64_t n, uint32_t D, uint32_t S_eff,
                             const uint64_t *bounds, uint32_t model, float *vals_out);

int drref_curvefit_decode_seg(const float *coef, const uint32_t *sigma, uint64_t n, uint32_t D, uint32_t S_eff,
                              const uint64_t *bounds, float *vals_out)
{
    return drref_curvefit_decode_ex(coef, sigma, n, D, S_eff, bounds, DRREF_FIT_POLY, vals_out);
}

/*
 * Decoder for either model: a DEXP run's value at abscissa t is
 * a e^(b t) + c e^(d t) in double on the fp32 row (a, b, c, d), rounded to
 * fp32 (D is 3 for DEXP records).
 */
int drref_curvefit_decode_ex(const float *coef, const uint32_t *sigma, uint64_t n, uint32_t D, uint32_t S_eff,
                             const uint64_t *bounds, uint32_t model, float *vals_out)
{
    if (model > DRREF_FIT_DEXP)
        return DRREF_EINVAL;
    if ((!coef || !sigma || !vals_out || !bounds) && n)
        return DRREF_EINVAL;
    if (D > DRREF_MAX_DEG || (n && S_eff < 1))
        return DRREF_EINVAL;
    if (n == 0)
        return DRREF_OK;
    if (bounds[0] != 0 || bounds[S_eff] != n)
        return DRREF_EINVAL;
    for (uint32_t s = 0; s < S_eff; ++s)
        if (bounds[s + 1] <= bounds[s])
            return DRREF_EINVAL;
    const uint32_t D_eff = n >= (uint64_t)D + 1 ? D : (uint32_t)(n - 1);
    const uint32_t b = drref_sigma_bits(n);
    for (uint64_t q = 0; q < n; ++q) {
        const uint64_t rank = sigma_get(sigma, q, b);
        if (rank >= n)
            return DRREF_EINVAL;
        uint32_t s = 0;
        while (s + 1 < S_eff && bounds[s + 1] <= rank)
            ++s;
        const uint64_t lo = bounds[s], hi = bounds[s + 1];
        const double t = abscissa(rank - lo, hi - lo);
        const float *c = coef + (uint64_t)s * (D + 1);
        double y;
        if (model == DRREF_FIT_DEXP) {
            y = (double)c[0] * exp((double)c[1] * t) + (double)c[2] * exp((double)c[3] * t);
        } else {
            y = (double)c[D_eff];
            for (int p = (int)D_eff - 1; p >= 0; --p)
                y = y * t + (double)c[p];
        }
        vals_out[q] = (float)y;
    }
    return DRREF_OK;
}

int drref_curvefit_decode(const float *coef, const uint32_t *sigma, uint64_t n, uint32_t D, uint32_t S,
                          float *vals_out)
{
    if ((!coef || !sigma || !vals_out) && n)
        return DRREF_EINVAL;
    if (D > DRREF_MAX_DEG || S < 1)
        return DRREF_EINVAL;
    if (n == 0)
        return DRREF_OK;
    uint32_t S_eff, D_eff;
    drref_fit_shape(n, D, S, &S_eff, &D_eff);
    uint32_t b = drref_sigma_bits(n);
    for (uint64_t q = 0; q < n; ++q) {
        uint64_t rank = sigma_get(sigma, q, b);
        if (rank >= n)
            return DRREF_EINVAL;
        uint32_t s = 0;
        while (s + 1 < S_eff && seg_lo(s + 1, n, S_eff) <= rank)
            ++s;
        uint64_t lo = seg_lo(s, n, S_eff), hi = seg_lo(s + 1, n, S_eff);
        double t = abscissa(rank - lo, hi - lo);
        const float *c = coef + (uint64_t)s * (D + 1);
        double y = (double)c[D_eff];
        for (int p = (int)D_eff - 1; p >= 0; --p)
            y = y * t + (double)c[p];
        vals_out[q] = (float)y;
    }
    return DRREF_OK;
}

/* ------------------------------------------------------------------------ */
/* Index policies (Section 4; Sections 10.4 and 10.5).                       */
/* ------------------------------------------------------------------------ */

/*
 * Policy P0 keeps every positive of the query (Section 4, "No-error
 * approach").  The other policies keep r of the |P| positives, so that only
 * r values are sent: policy P1 picks them at random (Section 4, "Random
 * approach"; Section 10.5), the deterministic policies of Section 10.4 take
 * the leftmost, middle or rightmost r of P in index order.
 *
 * Sender and receiver must pick the same r positives without exchanging
 * them.  Both run the same query, so P is the same on both sides, and P1 is
 * made reproducible by a keyed pseudo-random permutation pi of the ranks
 * [0, |P|) that both evaluate: the positive of rank q is kept iff
 * pi(q) < r, and its value is value number pi(q).  For the deterministic
 * policies the value number is the rank within the kept run.  (The paper
 * leaves the source of randomness open; this keyed permutation is this
 * codec's reading.)
 *
 * pi is a 4-round Feistel network on 2h-bit words (h = ceil(ceil(log2 N)/2),
 * at least 1), with round function F_j(x) = MurmurHash3_x86_32 of the
 * 4-byte little-endian x with seed (seed + j), reduced to h bits, and cycle
 * walking (Black and Rogaway, "Ciphers with arbitrary finite domains",
 * CT-RSA 2002) to stay inside [0, N): the network is applied again until
 * the value falls below N.  A Feistel network is a bijection of the 2h-bit
 * words for any round function, and cycle walking restricts a bijection to
 * a bijection of [0, N).
 */
#define DRREF_POLICY_P0 0u
#define DRREF_POLICY_RANDOM 1u
#define DRREF_POLICY_LEFTMOST 2u
#define DRREF_POLICY_MIDDLE 3u
#define DRREF_POLICY_RIGHTMOST 4u
#define DRREF_NO_SLOT 0xffffffffu

static uint32_t feistel_round(uint32_t x, uint32_t seed, uint32_t j, uint32_t mask)
{
    uint8_t le[4] = {(uint8_t)(x & 0xff), (uint8_t)((x >> 8) & 0xff), (uint8_t)((x >> 16) & 0xff),
                     (uint8_t)((x >> 24) & 0xff)};
    return drref_murmur3_32(le, 4, seed + j) & mask;
}

static uint32_t feistel(uint32_t x, uint32_t h, uint32_t seed)
{
    const uint32_t mask = (h >= 32) ? 0xffffffffu : ((1u << h) - 1u);
    uint32_t L = (x >> h) & mask, R = x & mask;
    for (uint32_t j = 0; j < 4; ++j) {
        uint32_t t = L ^ feistel_round(R, seed, j, mask);
        L = R;
        R = t;
    }
    return (L << h) | R;
}

/* half width h for a domain of N values: 2h >= ceil(log2 N), h >= 1 */
static uint32_t feistel_half(uint64_t N)
{
    uint32_t bits = 0;
    while (bits < 32 && (1ull << bits) < N) ++bits;
    uint32_t h = (bits + 1) / 2;
    return h < 1 ? 1 : h;
}

/* pi(q) for q < N (N >= 1, N <= 2^32) */
uint32_t drref_perm(uint32_t q, uint64_t N, uint32_t seed)
{
    const uint32_t h = feistel_half(N);
    uint32_t y = q;
    do {
        y = feistel(y, h, seed);
    } while ((uint64_t)y >= N);
    return y;
}

/*
 * For each rank q of the |P| = npos positives: the value number it gets, or
 * DRREF_NO_SLOT if the policy drops it.  The number of kept positives goes to
 * *ncoded (npos for P0, min(r, npos) otherwise).
 */
int drref_policy_slots(uint64_t npos, uint64_t r, uint32_t policy, uint32_t seed, uint32_t *slot_out,
                       uint64_t *ncoded)
{
    if (policy > DRREF_POLICY_RIGHTMOST || npos > 0xffffffffull) return DRREF_EINVAL;
    const uint64_t keep = policy == DRREF_POLICY_P0 ? npos : (r < npos ? r : npos);
    *ncoded = keep;
    const uint64_t mid0 = (npos - keep) / 2, right0 = npos - keep;
    for (uint64_t q = 0; q < npos; ++q) {
        uint64_t slot = DRREF_NO_SLOT;
        switch (policy) {
        case DRREF_POLICY_P0:
            slot = q;
            break;
        case DRREF_POLICY_RANDOM: {
            const uint32_t p = drref_perm((uint32_t)q, npos, seed);
            if (p < keep) slot = p;
            break;
        }
        case DRREF_POLICY_LEFTMOST:
            if (q < keep) slot = q;
            break;
        case DRREF_POLICY_MIDDLE:
            if (q >= mid0 && q < mid0 + keep) slot = q - mid0;
            break;
        default: /* rightmost */
            if (q >= right0) slot = q - right0;
            break;
        }
        slot_out[q] = (uint32_t)slot;
    }
    return DRREF_OK;
}
