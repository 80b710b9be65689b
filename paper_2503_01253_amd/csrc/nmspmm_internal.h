// Helpers shared by the two halves of the library (host packer and device
// dispatch).  Not part of the public ABI.
#ifndef NMSPMM_INTERNAL_H
#define NMSPMM_INTERNAL_H

#include <cstdint>

namespace nmspmm {

// Shape rules of Sec. II-A without padding: k % M == 0, n % V == 0,
// 1 <= N <= M <= 256 (offsets fit a byte), V >= 1, no negative size.
bool shape_ok(int64_t m, int64_t n, int64_t k, int N, int M, int V);

// True when m*k, m*n and k*n fit comfortably in int64 element counts.
bool sizes_fit(int64_t m, int64_t n, int64_t k);

}  // namespace nmspmm

#endif
