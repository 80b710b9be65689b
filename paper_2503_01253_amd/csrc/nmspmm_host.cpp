// Host half of the C ABI: shape rules, size helpers, the offline packer and
// the pattern validator (Sec. II-A; the offline pre-processing of Sec. III-C.1).
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <limits>
#include <thread>
#include <vector>

#include "nmspmm.h"
#include "nmspmm_internal.h"

namespace nmspmm {

bool shape_ok(int64_t m, int64_t n, int64_t k, int N, int M, int V)
{
    if (m < 0 || n < 0 || k < 0) return false;
    if (M < 1 || M > 256 || N < 1 || N > M || V < 1) return false;
    return k % M == 0 && n % V == 0;
}

bool sizes_fit(int64_t m, int64_t n, int64_t k)
{
    const int64_t lim = std::numeric_limits<int64_t>::max() / 8;
    if (m && k > lim / m) return false;
    if (m && n > lim / m) return false;
    if (k && n > lim / k) return false;
    return true;
}

}  // namespace nmspmm

using namespace nmspmm;

extern "C" int64_t nmspmm_bc_elems(int64_t k, int64_t n, int N, int M)
{
    if (!shape_ok(0, n, k, N, M, 1) || !sizes_fit(1, n, k)) return -1;
    return (k / M) * N * n;
}

extern "C" int64_t nmspmm_idx_bytes(int64_t k, int64_t n, int N, int M, int V)
{
    if (!shape_ok(0, n, k, N, M, V) || !sizes_fit(1, n, k)) return -1;
    return (k / M) * N * (n / V);
}

extern "C" nmspmm_status_t nmspmm_compress(const float *B_dense, int64_t k, int64_t n,
                                           int N, int M, int V, float *Bc, uint8_t *idx)
{
    if (!shape_ok(0, n, k, N, M, V)) return NMSPMM_ERR_INVALID_ARG;
    if (!sizes_fit(1, n, k)) return NMSPMM_ERR_UNSUPPORTED;
    if (k == 0 || n == 0) return NMSPMM_OK;
    if (!B_dense || !Bc || !idx) return NMSPMM_ERR_INVALID_ARG;

    const int64_t groups = k / M, blocks = n / V, pairs = groups * blocks;
    // (window, column block) pairs are independent; split them over threads.
    auto pack_range = [=](int64_t lo, int64_t hi) {
        for (int64_t pair = lo; pair < hi; ++pair) {
            const int64_t g = pair / blocks, b = pair % blocks;
            const float *win = B_dense + g * M * n + b * V;
            // Squared L2 norm of each length-V row-vector.  fp32 squares are exact
            // in fp64 and the columns are added left to right, so the score (and
            // therefore every tie) is reproducible bit for bit.
            double norm2[256];
            int order[256];
            for (int o = 0; o < M; ++o) {
                const float *v = win + (int64_t)o * n;
                double s = 0.0;
                for (int c = 0; c < V; ++c) s += (double)v[c] * (double)v[c];
                norm2[o] = s;
                order[o] = o;
            }
            // Largest norms first, equal norms in offset order; keep the first N.
            std::stable_sort(order, order + M, [&](int x, int y) { return norm2[x] > norm2[y]; });
            std::sort(order, order + N);
            for (int r = 0; r < N; ++r) {
                const int64_t u = g * N + r;
                idx[u * blocks + b] = (uint8_t)order[r];
                std::memcpy(Bc + u * n + b * V, win + (int64_t)order[r] * n, sizeof(float) * (size_t)V);
            }
        }
    };
    const int64_t work = pairs * (int64_t)M * V;
    const int64_t nthreads = std::max<int64_t>(
        1, std::min<int64_t>({(int64_t)std::thread::hardware_concurrency(), 16, work / (1 << 20) + 1}));
    if (nthreads == 1) {
        pack_range(0, pairs);
    } else {
        std::vector<std::thread> pool;
        for (int64_t t = 0; t < nthreads; ++t)
            pool.emplace_back(pack_range, pairs * t / nthreads, pairs * (t + 1) / nthreads);
        for (auto &th : pool) th.join();
    }
    return NMSPMM_OK;
}

extern "C" nmspmm_status_t nmspmm_validate_idx(const uint8_t *idx, int64_t k, int64_t n,
                                               int N, int M, int V)
{
    if (!shape_ok(0, n, k, N, M, V)) return NMSPMM_ERR_INVALID_ARG;
    if (!sizes_fit(1, n, k)) return NMSPMM_ERR_UNSUPPORTED;
    const int64_t w = (k / M) * N, q = n / V;
    if (w * q == 0) return NMSPMM_OK;
    if (!idx) return NMSPMM_ERR_INVALID_ARG;
    for (int64_t u = 0; u < w; ++u) {
        const bool first_of_group = (u % N) == 0;
        for (int64_t b = 0; b < q; ++b) {
            const int cur = idx[u * q + b];
            if (cur >= M) return NMSPMM_ERR_INVALID_ARG;
            if (!first_of_group && cur <= idx[(u - 1) * q + b]) return NMSPMM_ERR_INVALID_ARG;
        }
    }
    return NMSPMM_OK;
}

extern "C" const char *nmspmm_status_string(nmspmm_status_t s)
{
    switch (s) {
    case NMSPMM_OK: return "ok";
    case NMSPMM_ERR_INVALID_ARG: return "invalid argument";
    case NMSPMM_ERR_UNSUPPORTED: return "unsupported request";
    case NMSPMM_ERR_HIP: return "HIP runtime error";
    case NMSPMM_ERR_SCRATCH:
        return "the shape needs more scratch than nmspmm_run_noalloc's static array holds "
               "(NMSPMM_NOALLOC_SCRATCH_BYTES); call nmspmm_run_ws with a workspace instead";
    }
    return "unknown status";
}
