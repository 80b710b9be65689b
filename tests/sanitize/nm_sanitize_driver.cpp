// Host-side sanitizer run (AddressSanitizer + UndefinedBehaviorSanitizer) of
// the CPU oracle (oracle/nm_oracle.c) and of the library's host half
// (csrc/nmspmm_host.cpp: packer, validator, size helpers), built from source
// with -fsanitize=address,undefined by tests/test_sanitizers.py.  Test code:
// it drives both, and checks them against each other and against a dense
// brute-force product; any out-of-bounds access, leak or undefined behaviour
// aborts the run.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "nmspmm.h"

extern "C" {
int oracle_spmm(const float *A, const float *Bc, const uint8_t *idx, double *C, int64_t m, int64_t n, int64_t k,
                int N, int M, int V);
int oracle_bound(const float *A, const float *Bc, const uint8_t *idx, double *Bnd, int64_t m, int64_t n,
                 int64_t k, int N, int M, int V);
int oracle_compress(const float *B, int64_t k, int64_t n, int N, int M, int V, float *Bc, uint8_t *idx);
int oracle_decompress(const float *Bc, const uint8_t *idx, int64_t k, int64_t n, int N, int M, int V, float *B);
int oracle_validate(const uint8_t *idx, int64_t k, int64_t n, int N, int M, int V);
int oracle_epilogue(double *C, int64_t m, int64_t n, double alpha, const float *bias, int act);
int oracle_dense(const float *A, const float *B, double *C, int64_t m, int64_t n, int64_t k);
int oracle_confusion(const double *Cs, const double *C, double *W, int64_t m, int64_t n);
}

namespace {

uint64_t g_state = 0x243f6a8885a308d3ull;

uint64_t next_u64()  // splitmix64
{
    uint64_t z = (g_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

float uniform() { return (float)((double)(next_u64() >> 11) * (1.0 / 9007199254740992.0) * 2.0 - 1.0); }

int failures = 0;

void expect(bool ok, const char *what, int64_t k, int64_t n, int N, int M, int V)
{
    if (!ok) {
        std::printf("FAIL %s at k=%lld n=%lld %d:%d V=%d\n", what, (long long)k, (long long)n, N, M, V);
        ++failures;
    }
}

// One shape: a random pruned B (N random kept rows per window and block), both
// packers, the round trip, the product against a dense brute force, the
// bound, the validators on good and corrupted offsets, the epilogue.
void run_case(int64_t m, int64_t k, int64_t n, int N, int M, int V, bool dense_input)
{
    const int64_t G = k / M, q = n / V, w = G * N;
    std::vector<float> B((size_t)(k * n), 0.f), A((size_t)(m * k));
    for (auto &a : A) a = uniform();
    for (int64_t g = 0; g < G; ++g)
        for (int64_t b = 0; b < q; ++b) {
            std::vector<int> rows(M);
            for (int o = 0; o < M; ++o) rows[o] = o;
            for (int o = M - 1; o > 0; --o) std::swap(rows[o], rows[next_u64() % (uint64_t)(o + 1)]);
            for (int r = 0; r < (dense_input ? M : N); ++r)
                for (int64_t c = b * V; c < (b + 1) * V; ++c) {
                    float v = uniform();
                    if (v == 0.f) v = 0.5f;
                    B[(size_t)((g * M + rows[r]) * n + c)] = v;
                }
        }
    std::vector<float> Bc_o((size_t)(w * n)), Bc_l((size_t)(w * n));
    std::vector<uint8_t> idx_o((size_t)(w * q)), idx_l((size_t)(w * q));
    expect(oracle_compress(B.data(), k, n, N, M, V, Bc_o.data(), idx_o.data()) == 0, "oracle_compress", k, n, N, M, V);
    expect(nmspmm_compress(B.data(), k, n, N, M, V, Bc_l.data(), idx_l.data()) == NMSPMM_OK, "nmspmm_compress", k,
           n, N, M, V);
    expect(std::memcmp(Bc_o.data(), Bc_l.data(), Bc_o.size() * sizeof(float)) == 0 &&
               std::memcmp(idx_o.data(), idx_l.data(), idx_o.size()) == 0,
           "packers agree byte for byte", k, n, N, M, V);
    expect(oracle_validate(idx_o.data(), k, n, N, M, V) == 0, "oracle_validate", k, n, N, M, V);
    expect(nmspmm_validate_idx(idx_o.data(), k, n, N, M, V) == NMSPMM_OK, "nmspmm_validate_idx", k, n, N, M, V);
    if (w > 0 && q > 0 && M < 256) {   // at M = 256 every byte is a valid offset
        std::vector<uint8_t> bad = idx_o;
        bad[0] = (uint8_t)M;
        expect(oracle_validate(bad.data(), k, n, N, M, V) == 2, "oracle_validate >= M", k, n, N, M, V);
        expect(nmspmm_validate_idx(bad.data(), k, n, N, M, V) == NMSPMM_ERR_INVALID_ARG, "validate >= M", k, n, N,
               M, V);
    }
    if (w > 1 && q > 0 && N > 1) {     // a repeated offset inside one window
        std::vector<uint8_t> bad = idx_o;
        bad[(size_t)q] = bad[0];
        expect(oracle_validate(bad.data(), k, n, N, M, V) == 3, "oracle_validate repeat", k, n, N, M, V);
        expect(nmspmm_validate_idx(bad.data(), k, n, N, M, V) == NMSPMM_ERR_INVALID_ARG, "validate repeat", k, n,
               N, M, V);
    }
    std::vector<float> Bd((size_t)(k * n));
    expect(oracle_decompress(Bc_o.data(), idx_o.data(), k, n, N, M, V, Bd.data()) == 0, "decompress", k, n, N, M, V);
    if (!dense_input) expect(std::memcmp(Bd.data(), B.data(), B.size() * sizeof(float)) == 0, "round trip", k, n, N, M, V);
    std::vector<double> C((size_t)(m * n)), Bnd((size_t)(m * n));
    expect(oracle_spmm(A.data(), Bc_o.data(), idx_o.data(), C.data(), m, n, k, N, M, V) == 0, "oracle_spmm", k, n, N,
           M, V);
    expect(oracle_bound(A.data(), Bc_o.data(), idx_o.data(), Bnd.data(), m, n, k, N, M, V) == 0, "oracle_bound", k, n,
           N, M, V);
    bool same = true;
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j) {
            double s = 0.0, sa = 0.0;
            for (int64_t kk = 0; kk < k; ++kk) {
                s += (double)A[(size_t)(i * k + kk)] * (double)Bd[(size_t)(kk * n + j)];
                sa += std::fabs((double)A[(size_t)(i * k + kk)] * (double)Bd[(size_t)(kk * n + j)]);
            }
            same = same && s == C[(size_t)(i * n + j)] && std::fabs(sa - Bnd[(size_t)(i * n + j)]) <= 1e-12 * sa;
        }
    expect(same, "product equals the dense brute force", k, n, N, M, V);
    std::vector<float> bias((size_t)n);
    for (auto &x : bias) x = uniform();
    // Eq. 2: the dense product of the decompressed (pruned) B equals the
    // sparse product, so W of the product against itself is zero
    std::vector<double> Cd((size_t)(m * n)), W((size_t)(m * n));
    expect(oracle_dense(A.data(), Bd.data(), Cd.data(), m, n, k) == 0, "oracle_dense", k, n, N, M, V);
    expect(oracle_confusion(C.data(), Cd.data(), W.data(), m, n) == 0, "oracle_confusion", k, n, N, M, V);
    bool zero = true;
    for (size_t e = 0; e < W.size(); ++e) zero = zero && W[e] == 0.0;
    expect(zero, "confusion of equal products is zero", k, n, N, M, V);
    for (int act = 0; act < 3; ++act)
        expect(oracle_epilogue(C.data(), m, n, 2.0, bias.data(), act) == 0, "oracle_epilogue", k, n, N, M, V);
}

}  // namespace

int main()
{
    // (m, k, n, N, M, V): offsets up to M = 256, ragged V, N = M, one window
    const int cases[][6] = {{5, 8, 12, 1, 4, 1},   {7, 16, 16, 2, 4, 4},    {3, 24, 10, 3, 8, 2},
                            {9, 64, 64, 16, 32, 32}, {4, 64, 32, 32, 32, 8}, {6, 35, 9, 5, 7, 3},
                            {1, 32, 64, 4, 32, 64},  {2, 512, 24, 5, 256, 8}, {3, 256, 256, 1, 256, 256},
                            {2, 32, 4096, 4, 32, 64}};
    for (const auto &c : cases)
        for (int dense = 0; dense < 2; ++dense) run_case(c[0], c[1], c[2], c[3], c[4], c[5], dense != 0);
    // large enough that the host packer splits its work over threads
    run_case(1, 2048, 2048, 8, 32, 32, false);
    // argument errors and empty shapes
    expect(nmspmm_compress(nullptr, 0, 64, 4, 32, 32, nullptr, nullptr) == NMSPMM_OK, "k == 0", 0, 64, 4, 32, 32);
    expect(nmspmm_compress(nullptr, 64, 60, 4, 32, 32, nullptr, nullptr) == NMSPMM_ERR_INVALID_ARG, "n % V", 64, 60, 4,
           32, 32);
    expect(nmspmm_bc_elems(4096, 4096, 16, 32) == 2048 * 4096, "bc_elems", 4096, 4096, 16, 32, 32);
    expect(nmspmm_idx_bytes(4096, 4096, 16, 32, 32) == 2048 * 128, "idx_bytes", 4096, 4096, 16, 32, 32);
    expect(nmspmm_bc_elems(INT64_MAX / 2, INT64_MAX / 2, 1, 1) == -1, "overflowing sizes", 0, 0, 1, 1, 1);
    expect(std::strlen(nmspmm_status_string((nmspmm_status_t)99)) > 0, "status string", 0, 0, 0, 0, 0);
    if (failures) {
        std::printf("%d FAILURES\n", failures);
        return 1;
    }
    std::printf("ALL OK\n");
    return 0;
}
