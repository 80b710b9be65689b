/*
 * nmspmm.h -- C ABI of the MI355X (gfx950) vector-wise N:M sparse matrix
 * multiplication library (NM-SpMM, arXiv 2503.01253).
 *
 * Problem (Sec. II-A): C = A * B with A m x k, B k x n, C m x n, all fp32,
 * row-major.  B is pruned with vector-wise N:M sparsity: inside every window
 * of M consecutive k-rows, N rows are kept, and one kept set is shared by each
 * block of V adjacent columns (the paper's vector length L).  B is stored
 * compressed as
 *   Bc  : w x n fp32, row-major, w = (k/M)*N            (the paper's B')
 *   idx : w x q uint8, row-major, q = n/V                (the paper's D)
 * where compressed row u = g*N + r (group g, r-th kept row) holds the kept
 * row-vector of window g for each column block b, and idx[u][b] is that row's
 * offset in [0, M) inside window g.  Offsets of one (g, b) are strictly
 * increasing.  The product computed is Eq. 1 read as
 *   C[i][j] = sum_{u<w} A[i][floor(u/N)*M + idx[u][floor(j/V)]] * Bc[u][j]
 * with no M/N rescaling (nmspmm_run_ex with alpha = M/N applies Eq. 1's
 * factor).
 *
 * Every entry point is extern "C", returns a status code and never throws.
 * The library's only global state is the static scratch array of
 * nmspmm_run_noalloc (with its per-device address) and a table of at most 16
 * cached workspaces of nmspmm_run and nmspmm_run_ex, one per (device,
 * stream), allocated on first use and kept until the process ends; it is
 * safe to call from several host threads.
 */
#ifndef NMSPMM_H
#define NMSPMM_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#if defined(__GNUC__)
#define NMSPMM_API __attribute__((visibility("default")))
#else
#define NMSPMM_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    NMSPMM_OK = 0,
    /* null pointer where data is required, negative size, k % M != 0,
     * n % V != 0, N < 1, N > M, M > 256, V < 1, or an idx entry that breaks
     * the pattern rules (nmspmm_validate_idx only) */
    NMSPMM_ERR_INVALID_ARG = 1,
    /* a well-formed request outside what the library implements (e.g. a
     * pointer not aligned to 4 bytes for an fp32 array, or sizes whose
     * products overflow int64) */
    NMSPMM_ERR_UNSUPPORTED = 2,
    /* the HIP runtime reported an error while launching */
    NMSPMM_ERR_HIP = 3,
    /* nmspmm_run_noalloc only: the shape's kernels need more scratch than
     * its static array holds (NMSPMM_NOALLOC_SCRATCH_BYTES); nothing ran */
    NMSPMM_ERR_SCRATCH = 4
} nmspmm_status_t;

/* Size of the static device scratch array of nmspmm_run_noalloc: 16 MiB per
 * device, enough for the direct-gather kernel's transposed A and offsets up
 * to 128 rows at k = n = 16384 (4:32, V = 64). */
#define NMSPMM_NOALLOC_SCRATCH_BYTES (16u << 20)

/* Number of fp32 elements of Bc, (k/M)*N*n, or -1 if (k, n, N, M) is invalid
 * (Sec. II-A: w = k*N/M rows). */
NMSPMM_API int64_t nmspmm_bc_elems(int64_t k, int64_t n, int N, int M);

/* Number of bytes of idx, (k/M)*N*(n/V), or -1 if the shape is invalid
 * (Sec. II-A: D is w x q; one uint8 per entry, enough for the log2(M) bits
 * of Sec. III-B.1 as long as M <= 256). */
NMSPMM_API int64_t nmspmm_idx_bytes(int64_t k, int64_t n, int N, int M, int V);

/* Offline packing (Sec. II-A; the offline pre-processing of Sec. III-C.1).
 * HOST pointers.  B_dense: k x n fp32 row-major, read only.  Bc and idx are
 * caller-allocated with nmspmm_bc_elems / nmspmm_idx_bytes entries.
 * For every (window g, column block b) the N row-vectors of largest squared
 * L2 norm over the block's V columns are kept (ties to the smaller offset),
 * their offsets written to idx in increasing order and their values copied to
 * Bc.  On an already pruned B whose kept values are non-zero this recovers
 * the kept set exactly.  k == 0 or n == 0 is a valid no-op.
 * Errors: NMSPMM_ERR_INVALID_ARG for a bad shape or a null pointer with a
 * non-empty output; nothing is written then. */
NMSPMM_API nmspmm_status_t nmspmm_compress(const float *B_dense, int64_t k, int64_t n,
                                int N, int M, int V, float *Bc, uint8_t *idx);

/* The sparse product (Eq. 1 as read above; Sec. III describes the tiled GPU
 * algorithm).  DEVICE pointers, all on the current HIP device.
 *   A  : m x k fp32 row-major (read only)
 *   Bc : w x n fp32 row-major (read only)
 *   idx: w x q uint8 row-major (read only)
 *   C  : m x n fp32 row-major, overwritten (must not alias the inputs)
 * Asynchronous on `stream` (NULL = the legacy default stream): the call
 * validates its arguments, enqueues the kernel(s) and returns; it does not
 * synchronize.  Kernel faults surface at the caller's next synchronization.
 * Workspace: where nmspmm_run_ws would run the direct-gather kernel (the
 * "+prep" names of nmspmm_kernel_name_ws), the call takes that kernel's
 * workspace from a buffer the library keeps for `stream` on the current
 * device (hipMalloc on the first call that needs it, and again, larger, on
 * a call that needs more; the call's kernels are ordered after the buffer's
 * previous use by an event), and the result is bit-identical to
 * nmspmm_run_ws's.  Up to 16 such buffers are kept; a call on a further
 * stream releases the least recently used idle one.  Growing or releasing a
 * buffer waits for its last kernels and calls hipFree, which synchronizes
 * the device (a graph capture running on another thread in the global
 * capture mode fails then); callers that mind pass a workspace through
 * nmspmm_run_ws.  While `stream` is
 * being captured into a graph, or when no buffer can be had, it runs the
 * kernels that take none instead (named by
 * nmspmm_kernel_name_tuned with with_workspace = 0), as it does for every
 * other shape.  Callers that cannot allocate at all use nmspmm_run_noalloc.  m == 0 or n == 0 returns NMSPMM_OK without a launch;
 * k == 0 writes zeros to C.  Summation order: fp32 MFMA accumulation in an
 * order fixed by the kernel variant; when the variant splits k across
 * workgroups through atomics (the name from nmspmm_kernel_name ends in
 * "+zero,splitS" with S > 1) the partial tiles are added to C with fp32
 * atomics, so the last bits of C may differ between runs; through the
 * workspace ("+ws,splitS") they are summed in a fixed order.  idx contents are not validated on the device
 * (use nmspmm_validate_idx on the host); an offset >= M is clamped to M-1
 * so that every access stays inside A, and the result is then unspecified.
 * Errors: NMSPMM_ERR_INVALID_ARG (bad shape, null pointer with non-empty
 * data), NMSPMM_ERR_UNSUPPORTED (misaligned pointer), NMSPMM_ERR_HIP (the
 * launch failed). */
NMSPMM_API nmspmm_status_t nmspmm_run(const float *A, const float *Bc, const uint8_t *idx,
                           float *C, int64_t m, int64_t n, int64_t k, int N,
                           int M, int V, hipStream_t stream);

/* Activation of the output epilogue of nmspmm_run_ex. */
typedef enum {
    NMSPMM_ACT_NONE = 0,
    NMSPMM_ACT_RELU = 1,   /* max(0, y) */
    NMSPMM_ACT_GELU = 2    /* y * Phi(y) = 0.5 * y * (1 + erf(y / sqrt(2))), fp32 erff */
} nmspmm_act_t;

/* nmspmm_run with an output epilogue:
 *   C[i][j] = act(alpha * (A * B_pruned)[i][j] + bias[j])
 * alpha = M/N gives Eq. 1's leading factor (Sec. II-A), which nmspmm_run
 * leaves out; bias (n fp32 values, DEVICE pointer, may be NULL: no bias) and
 * act are the epilogue of a linear layer such as the Llama layers of
 * Sec. IV-A (not part of the paper's operator).  Arguments, layout,
 * asynchrony and errors as nmspmm_run, plus NMSPMM_ERR_INVALID_ARG for an
 * unknown act and NMSPMM_ERR_UNSUPPORTED for a bias not aligned to 4 bytes.
 * The epilogue is applied once per output, in fp32, after the whole sum over
 * k (when the kernel splits k, by a second pass over C).  With alpha = 1,
 * bias = NULL and NMSPMM_ACT_NONE the result is bit-identical to
 * nmspmm_run. */
NMSPMM_API nmspmm_status_t nmspmm_run_ex(const float *A, const float *Bc, const uint8_t *idx,
                              float *C, int64_t m, int64_t n, int64_t k, int N,
                              int M, int V, float alpha, const float *bias,
                              nmspmm_act_t act, hipStream_t stream);

/* Bytes of workspace that nmspmm_run_ws can use for a product of this shape,
 * with buffers aligned as the allocator returns them: 0 when the kernel
 * chosen for the shape takes none, -1 for a bad shape.  Two kinds of kernel
 * take one: the direct-gather kernel for products of 17 to 128 rows with
 * V a multiple of 32 (a transposed copy of A, k x R floats with R the
 * smallest of 16, 32, 64 and 128 that holds m; the gather offsets, 4*w*(n/V)
 * bytes; and partial strips when it splits k), and the pipelined streaming
 * kernel when it splits k (its partial tiles).  Host only, no GPU call. */
NMSPMM_API int64_t nmspmm_workspace_bytes(int64_t m, int64_t n, int64_t k, int N, int M, int V);

/* nmspmm_run_ex with a caller-provided workspace (the same product, Eq. 1
 * as read above, and the same epilogue).
 *   workspace: DEVICE memory, 256-byte aligned, contents irrelevant, owned
 *              by the caller.
 *   workspace_bytes: its size.  When it is at least nmspmm_workspace_bytes
 *              for the shape, the call runs the kernels that use it:
 *              - short products: a first kernel writes A transposed and the
 *                gather offsets of D into the workspace, and the
 *                direct-gather kernel reads them;
 *              - a launch that splits k stores each workgroup's partial
 *                tile there, and a last kernel sums the partial tiles of
 *                every output in a fixed order and applies the epilogue.
 *              Either way: no zero fill of C, no atomics, and the result
 *              does not vary between runs.  Otherwise (NULL, smaller, or a
 *              shape whose kernel takes none) the call runs exactly as
 *              nmspmm_run_ex (which takes its cached workspace where
 *              the shape's kernel is the direct-gather kernel).
 * A workspace serves one call at a time: calls that overlap on one workspace
 * (on different streams) race.  Arguments, asynchrony and errors otherwise
 * as nmspmm_run_ex, plus NMSPMM_ERR_UNSUPPORTED for a workspace not aligned
 * to 256 bytes; with a large enough workspace the library allocates
 * nothing. */
NMSPMM_API nmspmm_status_t nmspmm_run_ws(const float *A, const float *Bc, const uint8_t *idx,
                              float *C, int64_t m, int64_t n, int64_t k, int N,
                              int M, int V, float alpha, const float *bias,
                              nmspmm_act_t act, void *workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* nmspmm_compress on the GPU, for pruning on the fly (same selection rule,
 * same output bytes as the host call: for every window and column block the
 * N row-vectors of largest fp64 squared L2 norm, ties to the smaller offset,
 * offsets increasing).  DEVICE pointers, all on the current HIP device;
 * asynchronous on `stream`, allocates nothing.  B_dense: k x n fp32
 * row-major, read only.  Bc: w x n fp32 and idx: w x q uint8 (w = (k/M)*N,
 * q = n/V), overwritten.  k == 0 or n == 0 returns NMSPMM_OK without a
 * launch.  NaN inputs are outside the contract (the output is then
 * unspecified, every access still in bounds).  Errors:
 * NMSPMM_ERR_INVALID_ARG (bad shape, null pointer with non-empty data),
 * NMSPMM_ERR_UNSUPPORTED (a float pointer not aligned to 4 bytes, sizes
 * beyond int64), NMSPMM_ERR_HIP (the launch failed). */
NMSPMM_API nmspmm_status_t nmspmm_compress_device(const float *B_dense, int64_t k, int64_t n,
                                       int N, int M, int V, float *Bc, uint8_t *idx,
                                       hipStream_t stream);

/* Eq. 2 (Sec. II-A), the confusion matrix between the N:M output and the
 * dense output of the same A:
 *   W[i][j] = |C_sparse[i][j] - C_dense[i][j]| / (m*n)
 * where C_sparse is Eq. 1's output with its M/N factor (nmspmm_run_ex with
 * alpha = M/N) and C_dense the product of A with the unpruned B (for
 * instance nmspmm_run on the N = M compression of B, which keeps every row).
 * DEVICE pointers, all on the current HIP device, m x n fp32 row-major.  W is
 * overwritten and may be the same array as C_sparse or C_dense (in place);
 * any other overlap is not allowed.  Each W[i][j] is the fp64 quotient of
 * the fp64 difference by the fp64 value of m*n, rounded once to fp32 (the
 * fp32 inputs convert to fp64 exactly).  Asynchronous on `stream`, allocates
 * nothing; m == 0 or n == 0 returns NMSPMM_OK without a launch.  Errors:
 * NMSPMM_ERR_INVALID_ARG (negative size, null pointer with non-empty data),
 * NMSPMM_ERR_UNSUPPORTED (a pointer not aligned to 4 bytes, m*n beyond
 * int64), NMSPMM_ERR_HIP (the launch failed). */
NMSPMM_API nmspmm_status_t nmspmm_confusion(const float *C_sparse, const float *C_dense, float *W,
                                 int64_t m, int64_t n, hipStream_t stream);

/* Host check of the pattern rules (Sec. II-A): every (group, block) has N
 * offsets, each < M, strictly increasing.  HOST pointer, O(w*q).
 * Returns NMSPMM_OK or NMSPMM_ERR_INVALID_ARG. */
NMSPMM_API nmspmm_status_t nmspmm_validate_idx(const uint8_t *idx, int64_t k, int64_t n,
                                    int N, int M, int V);

/* Static, never-null description of a status code. */
NMSPMM_API const char *nmspmm_status_string(nmspmm_status_t s);

/* Name of the kernel variant nmspmm_run would launch for this shape outside
 * graph capture (the direct-gather kernel with its cached workspace where
 * nmspmm_kernel_name_ws names it), assuming buffers aligned as the
 * allocator returns them: "none" when nothing is
 * launched, "invalid" for a bad shape.  The string stays valid until the next
 * call from the same thread.  For benchmark and profile reports; it launches
 * nothing. */
NMSPMM_API const char *nmspmm_kernel_name(int64_t m, int64_t n, int64_t k, int N, int M, int V);

/* The same for nmspmm_run_ws with a workspace of nmspmm_workspace_bytes
 * bytes ("+prep": the transposition kernel runs first; "+ws": partial tiles
 * go through the workspace). */
NMSPMM_API const char *nmspmm_kernel_name_ws(int64_t m, int64_t n, int64_t k, int N, int M, int V);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * nmspmm_run_ws with its workspace in a static device array of
 * NMSPMM_NOALLOC_SCRATCH_BYTES instead of caller memory.  Same product (Eq. 1
 * as read above), same epilogue, same kernels and bit-identical results as
 * nmspmm_run_ws given a workspace of nmspmm_workspace_bytes.  The call
 * allocates nothing and calls no allocating routine; every device the
 * library runs on holds its own copy of the array from the library's load
 * until the process ends.  The array's device address is looked up on the
 * first call on each device (make that first call outside graph capture).
 * Every call on a device shares that device's array: calls that overlap on
 * one device (several streams or host threads) race and must be serialised
 * by the caller.  Each call rewrites every scratch byte its kernels read, so
 * the array's old contents never matter.  Errors: as nmspmm_run_ex, plus
 * NMSPMM_ERR_SCRATCH when nmspmm_workspace_bytes for the shape exceeds
 * NMSPMM_NOALLOC_SCRATCH_BYTES (checked before anything is launched) and
 * NMSPMM_ERR_HIP when the array's address cannot be obtained. */
NMSPMM_API nmspmm_status_t nmspmm_run_noalloc(const float *A, const float *Bc, const uint8_t *idx,
                                   float *C, int64_t m, int64_t n, int64_t k, int N,
                                   int M, int V, float alpha, const float *bias,
                                   nmspmm_act_t act, hipStream_t stream);

/* ---- Tuning entry points: for tile sweeps and forced-variant tests only ----
 * The same product, Eq. 1 as read above, with the kernel choice overridden.
 * The default entry points above never read overrides (from the environment
 * or anywhere else); only these three take them, as an explicit string of
 * "KEY=VALUE" pairs separated by commas (NULL or "" = no override):
 *   TILE    tile name of the tiled kernel (e.g. "256x256m32w16"), or
 *           "skinny" for the streaming kernels of short products
 *   KA      stage depth of the tiled kernel: 32, 64 or 128 columns of A
 *   SPLITS  workgroups along k (any kernel that splits k)
 *   RT, SKCOLS, QPW            row tiles, columns per workgroup, quads per
 *                              wave of the register-operand streaming kernel
 *   PS      0: never the pipelined streaming kernel, 1: wherever it runs
 *   PSRT, PSBV, PSCPW, PSRB    its row tiles, columns per lane, column groups
 *                              per wave and ring rows
 *   GATHER  0: never the direct-gather kernel, 1: wherever it runs
 *   GCT, GNW, GD               its column tiles, waves and ring depth
 *   GH      1: one direct-gather workgroup per strip, 2: two row halves of
 *           64 rows each (above 64 rows, without split-k)
 *   RG      0: never the row-gather kernel, 1: wherever it runs (up to 32
 *           rows, V a multiple of 32)
 *   RGCT, RGNW, RGD            its column tiles, waves and ring depth
 * A request the kernels cannot honour falls back to another kernel (a
 * forced tile that does not fit the shape: the general kernel).  An
 * unknown key or a malformed pair makes the call fail with
 * NMSPMM_ERR_INVALID_ARG ("invalid" / -1 for the two queries).  Arguments,
 * layout, asynchrony, workspace rules and errors otherwise as
 * nmspmm_run_ws, except that without a large enough workspace the call runs
 * the kernels that take none (it takes no cached workspace). */
NMSPMM_API nmspmm_status_t nmspmm_run_tuned(const float *A, const float *Bc, const uint8_t *idx,
                                 float *C, int64_t m, int64_t n, int64_t k, int N,
                                 int M, int V, float alpha, const float *bias,
                                 nmspmm_act_t act, void *workspace, size_t workspace_bytes,
                                 const char *tuning, hipStream_t stream);

/* Under the overrides of `tuning`: the kernels nmspmm_run_tuned launches
 * without a workspace (with_workspace == 0; the tuned call takes no cached
 * workspace) or with one of nmspmm_workspace_bytes_tuned bytes (otherwise,
 * as nmspmm_kernel_name_ws). */
NMSPMM_API const char *nmspmm_kernel_name_tuned(int64_t m, int64_t n, int64_t k, int N, int M, int V,
                                     int with_workspace, const char *tuning);

/* nmspmm_workspace_bytes under the overrides of `tuning`. */
NMSPMM_API int64_t nmspmm_workspace_bytes_tuned(int64_t m, int64_t n, int64_t k, int N, int M, int V,
                                     const char *tuning);

#ifdef __cplusplus
}
#endif
#endif /* NMSPMM_H */
