/*
 * nm_oracle.c -- CPU reference ("oracle") for vector-wise N:M sparse matrix
 * multiplication, as defined in NM-SpMM (arXiv 2503.01253).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test suite, the smoke check of the build entry
 * point and the CPU-baseline leg of the benchmark use it.  It shares no code,
 * header, table or helper with the HIP library; the two are compared, never
 * combined.
 *
 * Everything here is deliberately plain: fp64 accumulation, loops in the
 * order of the definition, no blocking, no fusion, no reordering.  OpenMP
 * splits the work over output rows only, which does not change the order of
 * any addition.
 *
 * Notation (Sec. II-A): A is m x k, the pruned weight B is k x n, C = A * B is
 * m x n.  In every window ("group") of M consecutive k-rows, exactly N rows
 * are kept, and the kept set is shared by a block of V adjacent columns (the
 * paper calls V the vector length L).  G = k/M groups, w = G*N rows of the
 * compressed matrix Bc (the paper's B'), q = n/V column blocks.  idx (the
 * paper's D, w x q) holds, for compressed row u and column block b, the offset
 * of that kept row inside its window, in [0, M).
 *
 * Readings taken where the paper is garbled or silent (each is also listed in
 * the design notes of the repository):
 *  - Eq. 1 writes A's column as u*M/N + D[u][j/L].  Read as
 *    floor(u/N)*M + D[u][floor(j/V)]: D holds an offset inside window
 *    floor(u/N), so the window base must be the group index times M.
 *  - Eq. 1 sums u = 0..w; B' has w rows, so the sum runs over u = 0..w-1.
 *  - Eq. 1's leading factor M/N is not applied: the kernels of Sec. III
 *    accumulate plain products (the inner kernel of Sec. III-B), and the
 *    operator C = A (*) (B, D) is the product with the pruned B.
 *  - Offsets within one (group, block) are stored strictly increasing.
 *  - Eq. 2's C is the product with the unpruned B and its C' is Eq. 1's
 *    output with the factor M/N; W divides by m*n as printed.
 *  - The paper leaves the pruning rule to pruning algorithms (Sec. II-B); the
 *    compressor keeps the N rows of largest squared L2 norm over the block's
 *    V columns, ties going to the smaller offset.  On an already pruned
 *    matrix whose kept entries are non-zero this recovers the kept set.
 *
 * Pins (tests that tie this file to the mathematics, not to itself):
 *  - oracle_spmm equals, bit for bit, a dense sequential-k fp64 product with
 *    the pruned dense matrix (pruned terms add zeros; fp32 x fp32 products
 *    are exact in fp64; increasing offsets keep the addition order).
 *  - N == M reduces to a dense GEMM; A == I returns the pruned B exactly.
 *  - A power-of-two encoding makes each output the bit mask of the k-rows
 *    that fed it (Fig. 1's parameters N=2, M=4, V=4).
 *  - oracle_compress recovers the generator's mask and round-trips through
 *    oracle_decompress; oracle_bound equals |A| * |B_pruned| from a library
 *    matmul to fp64 rounding.
 *  - oracle_dense equals oracle_spmm bit for bit at N == M (every row kept,
 *    same order) and a library matmul to fp64 rounding.
 *  - oracle_confusion reproduces a hand-worked case, the closed form
 *    (M/N - 1) * |A * B| / (m*n) on an already pruned B, and zero at N == M.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Return 0 when the shape is one Eq. 1 defines without padding (Sec. II-A:
 * k divisible by M, n divisible by V, 1 <= N <= M, offsets fit a byte). */
int oracle_shape_ok(int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    if (m < 0 || n < 0 || k < 0) return 1;
    if (M < 1 || M > 256 || N < 1 || N > M || V < 1) return 1;
    if (k % M != 0 || n % V != 0) return 1;
    return 0;
}

/* Number of OpenMP threads a parallel region will use. */
int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_threads(int t)
{
#ifdef _OPENMP
    if (t > 0) omp_set_num_threads(t);
#else
    (void)t;
#endif
}

/* Eq. 1 (read as above), Sec. II-A:
 *   C[i][j] = sum_{u=0}^{w-1} A[i][floor(u/N)*M + idx[u][floor(j/V)]] * Bc[u][j]
 * accumulated in fp64 with u increasing for every (i, j). */
int oracle_spmm(const float *A, const float *Bc, const uint8_t *idx, double *C,
                int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    if (oracle_shape_ok(m, n, k, N, M, V)) return 1;
    const int64_t w = (k / M) * N, q = n / V;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double *c = C + i * n;
        const float *a = A + i * k;
        for (int64_t j = 0; j < n; ++j) c[j] = 0.0;
        for (int64_t u = 0; u < w; ++u) {
            const int64_t window = (u / N) * M;
            const float *brow = Bc + u * n;
            const uint8_t *drow = idx + u * q;
            for (int64_t b = 0; b < q; ++b) {
                const double av = (double)a[window + drow[b]];
                double *cb = c + b * V;
                const float *bb = brow + b * V;
                for (int64_t jj = 0; jj < V; ++jj) cb[jj] += av * (double)bb[jj];
            }
        }
    }
    return 0;
}

/* The magnitude bound used by the parity tolerance:
 *   Bound[i][j] = sum_u |A[i][floor(u/N)*M + idx[u][floor(j/V)]]| * |Bc[u][j]|
 * which equals sum_k |A[i][k]| |B_pruned[k][j]| because pruned entries are 0. */
int oracle_bound(const float *A, const float *Bc, const uint8_t *idx, double *Bnd,
                 int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    if (oracle_shape_ok(m, n, k, N, M, V)) return 1;
    const int64_t w = (k / M) * N, q = n / V;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double *c = Bnd + i * n;
        const float *a = A + i * k;
        for (int64_t j = 0; j < n; ++j) c[j] = 0.0;
        for (int64_t u = 0; u < w; ++u) {
            const int64_t window = (u / N) * M;
            const float *brow = Bc + u * n;
            const uint8_t *drow = idx + u * q;
            for (int64_t b = 0; b < q; ++b) {
                const double av = fabs((double)a[window + drow[b]]);
                double *cb = c + b * V;
                const float *bb = brow + b * V;
                for (int64_t jj = 0; jj < V; ++jj) cb[jj] += av * fabs((double)bb[jj]);
            }
        }
    }
    return 0;
}

/* Sec. II-A: from the dense B (k x n), keep N of every M consecutive
 * row-vectors of length V in each column block, store the kept vectors in Bc
 * (w x n) and their window offsets in idx (w x q), offsets ascending.
 * Selection: largest sum of squares over the block (fp64), ties to the
 * smaller offset. */
int oracle_compress(const float *B, int64_t k, int64_t n, int N, int M, int V,
                    float *Bc, uint8_t *idx)
{
    if (oracle_shape_ok(0, n, k, N, M, V)) return 1;
    const int64_t G = k / M, q = n / V;
    for (int64_t g = 0; g < G; ++g) {
        for (int64_t b = 0; b < q; ++b) {
            double score[256];
            int taken[256];
            for (int o = 0; o < M; ++o) {
                double s = 0.0;
                const float *row = B + (g * M + o) * n + b * V;
                for (int64_t c = 0; c < V; ++c) s += (double)row[c] * (double)row[c];
                score[o] = s;
                taken[o] = 0;
            }
            /* pick the N largest, one at a time; strict '>' keeps the
             * smaller offset on ties */
            for (int r = 0; r < N; ++r) {
                int best = -1;
                for (int o = 0; o < M; ++o) {
                    if (taken[o]) continue;
                    if (best < 0 || score[o] > score[best]) best = o;
                }
                taken[best] = 1;
            }
            /* emit in ascending offset order */
            int r = 0;
            for (int o = 0; o < M; ++o) {
                if (!taken[o]) continue;
                const int64_t u = g * N + r;
                idx[u * q + b] = (uint8_t)o;
                memcpy(Bc + u * n + b * V, B + (g * M + o) * n + b * V,
                       (size_t)V * sizeof(float));
                ++r;
            }
        }
    }
    return 0;
}

/* Inverse of the packing: scatter Bc back into a zeroed k x n matrix. */
int oracle_decompress(const float *Bc, const uint8_t *idx, int64_t k, int64_t n,
                      int N, int M, int V, float *B)
{
    if (oracle_shape_ok(0, n, k, N, M, V)) return 1;
    const int64_t w = (k / M) * N, q = n / V;
    memset(B, 0, (size_t)(k * n) * sizeof(float));
    for (int64_t u = 0; u < w; ++u) {
        const int64_t window = (u / N) * M;
        for (int64_t b = 0; b < q; ++b) {
            const int64_t row = window + idx[u * q + b];
            memcpy(B + row * n + b * V, Bc + u * n + b * V, (size_t)V * sizeof(float));
        }
    }
    return 0;
}

/* Pattern validity (Sec. II-A, Sec. III-B.1): every (group, block) holds N
 * offsets, each < M, strictly increasing.  Returns 0 if valid, 1 for a bad
 * shape, 2 for an offset >= M, 3 for a non-increasing pair. */
int oracle_validate(const uint8_t *idx, int64_t k, int64_t n, int N, int M, int V)
{
    if (oracle_shape_ok(0, n, k, N, M, V)) return 1;
    const int64_t G = k / M, q = n / V;
    for (int64_t g = 0; g < G; ++g) {
        for (int64_t b = 0; b < q; ++b) {
            for (int r = 0; r < N; ++r) {
                const int o = idx[(g * N + r) * q + b];
                if (o >= M) return 2;
                if (r > 0 && o <= idx[(g * N + r - 1) * q + b]) return 3;
            }
        }
    }
    return 0;
}

/* Output epilogue, in place on an fp64 product C (m x n):
 *   C[i][j] <- act(alpha * C[i][j] + bias[j])
 * alpha = M/N applies Eq. 1's leading factor (Sec. II-A), which the product
 * above leaves out.  The bias vector (n entries, may be NULL) and the
 * activation are the usual epilogue of a linear layer such as the Llama
 * layers of Sec. IV-A; the paper's operator itself has neither.
 * act: 0 none; 1 ReLU, max(0, y); 2 GELU, y * Phi(y) with Phi the standard
 * normal CDF, 0.5 * (1 + erf(y / sqrt(2))).  Returns 1 for an unknown act. */
int oracle_epilogue(double *C, int64_t m, int64_t n, double alpha, const float *bias, int act)
{
    if (act < 0 || act > 2) return 1;
    for (int64_t i = 0; i < m; ++i) {
        for (int64_t j = 0; j < n; ++j) {
            double y = alpha * C[i * n + j];
            if (bias) y += (double)bias[j];
            if (act == 1) y = y > 0.0 ? y : 0.0;
            else if (act == 2) y = 0.5 * y * (1.0 + erf(y / sqrt(2.0)));
            C[i * n + j] = y;
        }
    }
    return 0;
}

/* The dense product that Eq. 2 compares against (Sec. II-A): A (m x k) times
 * the unpruned B (k x n),
 *   C[i][j] = sum_{kk=0}^{k-1} A[i][kk] * B[kk][j]
 * accumulated in fp64 with kk increasing for every (i, j).  Returns 1 for a
 * negative size. */
int oracle_dense(const float *A, const float *B, double *C, int64_t m, int64_t n, int64_t k)
{
    if (m < 0 || n < 0 || k < 0) return 1;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double *c = C + i * n;
        const float *a = A + i * k;
        for (int64_t j = 0; j < n; ++j) c[j] = 0.0;
        for (int64_t kk = 0; kk < k; ++kk) {
            const double av = (double)a[kk];
            const float *brow = B + kk * n;
            for (int64_t j = 0; j < n; ++j) c[j] += av * (double)brow[j];
        }
    }
    return 0;
}

/* Eq. 2 (Sec. II-A), the confusion matrix between the N:M output Cs (Eq. 1
 * with its M/N factor, i.e. oracle_spmm followed by oracle_epilogue with
 * alpha = M/N) and the dense output C (oracle_dense), both m x n:
 *   W[i][j] = |Cs[i][j] - C[i][j]| / (m * n)
 * in fp64, m * n taken as an fp64 value.  Returns 1 for a negative size. */
int oracle_confusion(const double *Cs, const double *C, double *W, int64_t m, int64_t n)
{
    if (m < 0 || n < 0) return 1;
    const double mn = (double)m * (double)n;
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j) W[i * n + j] = fabs(Cs[i * n + j] - C[i * n + j]) / mn;
    return 0;
}
