/*
 * marlin.h - C ABI of the MI355X (gfx950) W4A16 GEMM library.
 *
 * The library computes the mixed-precision product of MARLIN
 * (arXiv 2408.11743, Section 3.4 "Kernel Design"):
 *
 *     C[m][n] = sum_k A[m][k] * s[k / g][n] * (q[k][n] - 8)
 *
 * A is fp16 [M][K] (row-major), q are unsigned 4-bit codes of a K x N weight
 * matrix quantised symmetrically with zero point 8 (Section 3.4,
 * "Dequantization and Tensor Cores"), s are fp16 scales, one per group of g
 * consecutive rows of K in each column or one per column (g = K), and C is
 * fp16 [M][N] (row-major).  Products accumulate in fp32; C is rounded to
 * fp16 (round to nearest even) once, at the end.
 *
 * Conventions for every entry point:
 *  - Pointers named as device pointers must be device memory (hipMalloc or a
 *    PyTorch CUDA tensor) of the current device; the library never
 *    allocates, frees or synchronises, and never reads host memory.
 *  - Work is enqueued asynchronously on `stream` (0 = the null stream).
 *  - Every argument check runs on the host before any HIP call; a failed
 *    check returns a status and enqueues nothing.
 *  - The caller owns all buffers.  Outputs must not alias inputs.
 *  - Shapes: K % 128 == 0, N % 64 == 0, K >= 128, N >= 64, M >= 0
 *    (M == 0 enqueues nothing and returns MARLIN_OK).  K, N <= 2^20,
 *    K * N < 2^32 (packed weights below 2 GiB), M <= 2^24.
 *  - Group size `group`: -1 or K (one scale per column), or a multiple of
 *    128 that divides K (e.g. 128).  G = K / group scale rows (1 per column
 *    for per-channel scales).
 *  - Alignment: all device pointers 16-byte aligned.
 */
#ifndef MARLIN_MI355X_H
#define MARLIN_MI355X_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MARLIN_OK = 0,
    MARLIN_ERR_NULL_POINTER = 1,      /* a required pointer is NULL                 */
    MARLIN_ERR_INVALID_SHAPE = 2,     /* M, N or K outside the constraints above    */
    MARLIN_ERR_UNSUPPORTED_GROUP = 3, /* group not in {-1, K, 128*j dividing K}     */
    MARLIN_ERR_MISALIGNED = 4,        /* a device pointer is not 16-byte aligned    */
    MARLIN_ERR_WORKSPACE_TOO_SMALL = 5, /* workspace_bytes < marlin_workspace_bytes */
    MARLIN_ERR_HIP = 6,               /* a HIP runtime call or launch failed        */
    MARLIN_ERR_INVALID_SPARSITY = 7,  /* reserved for the 2:4 entry points          */
    MARLIN_ERR_INVALID_ARGUMENT = 8   /* another argument out of its range          */
} marlin_status_t;

/* Version of the packed weight / scale layouts described below.  A packed
 * buffer is only valid for a library with the same layout version. */
#define MARLIN_LAYOUT_VERSION 1

/* Returns MARLIN_LAYOUT_VERSION of the library actually loaded. */
int marlin_layout_version(void);

/* Human-readable name of a status code (static storage, never NULL). */
const char *marlin_status_string(marlin_status_t status);

/* Bytes of the packed weights: K * N / 2 (4 bits per weight; the weights
 * are streamed exactly once per call, Section 3.4 "Maximizing Loading
 * Bandwidth").  Returns 0 for shapes that violate the constraints. */
size_t marlin_packed_weight_bytes(int64_t K, int64_t N);

/* Bytes of the packed scales: 2 * G * N.  Returns 0 for invalid arguments. */
size_t marlin_packed_scale_bytes(int64_t K, int64_t N, int64_t group);

/* Bytes of the workspace marlin_gemm (and marlin_gemm_sparse) needs for
 * this problem (arrival counters plus fp32 partial tiles of the Stream-K
 * style split, Section 3.4 "Striped Partitioning").  Pure host arithmetic:
 * it makes no HIP call and does not depend on the device (it is the size for
 * a 256-compute-unit device; on a device with fewer compute units, a launch
 * whose preferred split would need more is planned to fit it).  Memoised:
 * a repeated query is a table lookup.  Returns 0 for invalid arguments. */
size_t marlin_workspace_bytes(int64_t M, int64_t N, int64_t K, int64_t group);

/*
 * marlin_pack_weights - offline repack of codes and scales into the layout
 * the GEMM streams (Section 3.4: "Maximizing Loading Bandwidth" reshuffles
 * weight tiles so each thread issues one 16-byte load; "Dequantization and
 * Tensor Cores" orders each thread's codes for paired decoding; "Groups and
 * Instruction Ordering" reorganises the scales the same way).  Done once per
 * weight matrix; not on the timed path.
 *
 *   q        device, uint8 [K][N] row-major; only the low nibble of each byte
 *            is read (the code 0..15).
 *   s        device, fp16 bits [G][N] row-major.
 *   w_packed device, marlin_packed_weight_bytes(K, N) bytes, written.
 *   s_packed device, marlin_packed_scale_bytes(K, N, group) bytes, written.
 *
 * Packed weight layout (uint32 words; c = column tile of 64, ku = block of
 * 128 rows of K, nb = 16-column block in the tile, l = lane 0..63, t = 0..3):
 *
 *   word index  (((c * (K/128) + ku) * 4 + nb) * 64 + l) * 4 + t
 *   holds the 8 codes of column n = 64c + 16nb + (l % 16) and rows
 *   k = 128ku + 32t + 8(l / 16) + j, j = 0..7; code j sits in nibble
 *   p(j) = (j >> 1) + 4 * (j & 1), i.e. bits [4p, 4p + 4).
 *
 * so one 16-byte vector (t = 0..3) is a lane's operand for four 16x16x32
 * MFMA steps, and a 1 KiB run (l = 0..63) is one 16 x 128 block of W^T.
 *
 * Packed scale layout (fp16; r = scale row 0..G-1, lg = 0..3, nb = 0..3,
 * i = 0..3):
 *
 *   index  (((c * G + r) * 4 + lg) * 4 + nb) * 4 + i
 *   holds s[r][64c + 16nb + 4lg + i].
 *
 * Pack and unpack are exact inverses for codes 0..15 and any fp16 bits.
 * Errors: NULL_POINTER, INVALID_SHAPE, UNSUPPORTED_GROUP, MISALIGNED, HIP.
 */
marlin_status_t marlin_pack_weights(const uint8_t *q, const uint16_t *s,
                                    int64_t K, int64_t N, int64_t group,
                                    void *w_packed, void *s_packed,
                                    hipStream_t stream);

/*
 * marlin_unpack_weights - inverse of marlin_pack_weights (same arguments
 * and layouts, directions swapped).  q receives codes 0..15 (high nibble 0).
 */
marlin_status_t marlin_unpack_weights(const void *w_packed, const void *s_packed,
                                      int64_t K, int64_t N, int64_t group,
                                      uint8_t *q, uint16_t *s, hipStream_t stream);

/*
 * marlin_gemm - C = A * dequant(W) (Section 3.4).
 *
 *   A          device, fp16 [M][K] row-major, read only.
 *   w_packed   device, packed weights (marlin_pack_weights layout).
 *   s_packed   device, packed scales (marlin_pack_weights layout, same group).
 *   C          device, fp16 [M][N] row-major, written (every element).
 *   workspace  device, >= marlin_workspace_bytes(M, N, K, group) bytes.  Its
 *              first 1 MiB (arrival counters) must be zero before its
 *              first use (zero-fill the whole buffer once); every call
 *              leaves the counters at zero again, so one workspace serves
 *              any sequence of calls, of any shapes, issued in order on one
 *              stream, as long as it is large enough for each.  Calls that
 *              may overlap (different streams) need separate workspaces.
 *
 * Accumulation is fp32.  Group scales multiply each 128-row fp32 partial
 * product (stream kernel with row groups of up to 32 rows, tile kernel) or,
 * in the wide kernel that serves large batches and the stream and pair
 * kernels with 64-row groups, the fp16 weights before the product (one fp16 rounding per
 * weight, as Section 3.4's "Groups and Instruction Ordering" does);
 * per-channel scales multiply the final sum once.  Any M up to 4096
 * runs in one launch: the rows are cut into segments (32 or 64 rows for the
 * stream kernel, the tile's rows for the tile and wide kernels) and each segment repeats the
 * weight matrix's tiles in the striped partition, so all segments share one
 * work split and one combination step (Section 3.4, Striped Partitioning,
 * on batches well above 64).  Larger M runs as launches of 4096 rows.
 * Results are bitwise reproducible for a given device, shape and input.
 *
 * The launch configuration comes from a cost model of the device (see
 * marlin_describe).  For tuning and tests, the environment variable
 * MARLIN_FORCE_CONFIG="kind=<stream|tile|wide>,nb=<1|2|4|8>,whole=<0|1>,
 * grid=<n>,waves=<4|8>,nw=<4|8>,ks=<1|2|4>,mb=<1|2|4>" (any subset: kernel,
 * column blocks per tile (per wave for the tile and wide kernels), partition,
 * work-groups, stream-kernel waves per work-group (eight with mb=4: the
 * pair kernel), tile-kernel waves and 128-row blocks per stage,
 * stream-kernel 16-row blocks per row group)
 * overrides it where the shape allows,
 * read at every call (parsed again only when its text changes);
 * configurations are memoised per shape, device and override, so a repeated
 * call plans in a table lookup;
 * marlin_workspace_bytes follows the same override, so size the workspace
 * under the setting the calls will see.
 * Errors: NULL_POINTER, INVALID_SHAPE, UNSUPPORTED_GROUP, MISALIGNED,
 * WORKSPACE_TOO_SMALL, HIP.
 */
marlin_status_t marlin_gemm(const uint16_t *A, const void *w_packed,
                            const void *s_packed, uint16_t *C,
                            void *workspace, size_t workspace_bytes,
                            int64_t M, int64_t N, int64_t K, int64_t group,
                            hipStream_t stream);

/*
 * marlin_gemm_no_alloc - marlin_gemm without a workspace argument, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * serving loops and harnesses that forbid hipMalloc.  It allocates nothing
 * and frees nothing.
 *
 *   A, w_packed, s_packed, C, M, N, K, group, stream: as for marlin_gemm.
 *
 * Its workspace is a file-scope device array of the library, 33 MiB
 * (1 MiB of arrival counters, 32 MiB of fp32 partial tiles), which each
 * device the library runs on holds from the library's first use there until
 * the process ends.  Every call on a device shares that device's array:
 * calls that may overlap on one device (different streams, concurrent graph
 * replays) race and must be ordered by the caller.  A launch whose preferred
 * Stream-K split would need more partial-tile space than the array holds is
 * planned with the best configuration that fits (whole tiles need none), so
 * every shape marlin_gemm accepts runs; the result is then within the same
 * tolerance of the definition as marlin_gemm's, and bitwise reproducible.
 * The first call on a device looks up the array's address there and clears
 * its counters with a small kernel on `stream`, ahead of the call's own
 * launches; every call leaves the counters at zero.
 * Errors: NULL_POINTER, INVALID_SHAPE, UNSUPPORTED_GROUP, MISALIGNED, HIP,
 * and WORKSPACE_TOO_SMALL should a launch ever need more than the array
 * (none does: it is checked per launch before anything is enqueued).
 */
marlin_status_t marlin_gemm_no_alloc(const uint16_t *A, const void *w_packed, const void *s_packed,
                                     uint16_t *C, int64_t M, int64_t N, int64_t K, int64_t group,
                                     hipStream_t stream);

/*
 * marlin_describe - the launch configuration marlin_gemm would use for this
 * problem on the current device (or on a 256-CU device when no device is
 * visible), as one NUL-terminated line: the kernel's name with its template
 * arguments as a profiler reports it, then "cols=<columns per tile>
 * rg=<row groups> partition=<whole|streamk> grid=<work-groups>", for the
 * first launch (the first 4096 rows).  The stream kernel's template arguments are
 * <16-row blocks, 16-column blocks, ring depth, activation rows / 4, waves,
 * per-channel>, the tile kernel's <waves along N, waves along M, 16-row
 * blocks per wave, 16-column blocks per wave, 128-row blocks per stage,
 * per-channel>, the wide kernel's <16-row blocks per wave, 16-column blocks
 * per wave, ring depth, per-channel>.  Row groups are of 32 rows for the
 * stream kernel and of the tile's rows for the tile and wide kernels.  Pure
 * host code apart from
 * reading the device's compute-unit count; enqueues nothing.
 *
 *   buf        host, buf_bytes bytes, written (truncated to fit, always
 *              NUL-terminated when buf_bytes > 0).
 * Errors: NULL_POINTER (buf NULL), INVALID_SHAPE, UNSUPPORTED_GROUP.
 */
marlin_status_t marlin_describe(int64_t M, int64_t N, int64_t K, int64_t group,
                                char *buf, size_t buf_bytes);

/*
 * ---- 2:4 sparse weights (Section 4, "Sparse-MARLIN") ----
 *
 * The weight matrix is 2:4 sparse along K: in every group of 4 consecutive
 * rows of a column at most two weights are non-zero.  It is given as the
 * dense code matrix q [K][N] of marlin_pack_weights with the pruned
 * positions holding code 8 (weight s * (8 - 8) = 0), so the product is the
 * dense definition C = A * (s * (q - 8)) on that matrix.  The packed form
 * keeps two codes per group plus their 2-bit row indices, 3/8 byte per
 * weight instead of 1/2, and feeds v_smfmac_f32_16x16x64_f16.
 */

/* Bytes of the packed sparse weights: 3*K*N/8 (0 for an invalid shape). */
size_t marlin_packed_sparse_weight_bytes(int64_t K, int64_t N);

/*
 * marlin_pack_sparse_weights - codes and scales -> the sparse packed layout.
 *
 *   q, s, K, N, group, s_packed, stream: as for marlin_pack_weights (s_packed
 *              has the same layout and size).
 *   w_packed   device, marlin_packed_sparse_weight_bytes(K, N) bytes, written.
 *
 * Kept rows: in each group of 4 rows of a column, the first two whose code
 * is not 8; a group with fewer is completed with its lowest rows of code 8.
 * So a matrix with at most two non-8 codes per group is represented
 * exactly; codes after the second non-8 code of a group are dropped (such a
 * matrix is not 2:4 sparse).
 *
 * Packed sparse layout (uint32 words; c = 64-column tile, ku = 128-row
 * block, nb = 16-column block, l = lane 0..63, h = 0..1, g = 0..3, t = 0..1),
 * unit (c, ku) at word (c*KU + ku)*768:
 *   codes: word ((d >> 2)*64 + l)*4 + (d & 3), d = 2*nb + h, holds the kept
 *     codes j = 2g + t of column n = 64c + 16nb + l%16 for the row groups
 *     128ku + 64h + 16(l/16) + 4g .. + 3, code j in nibble (j >> 1) + 4(j & 1);
 *   row indices: word 512 + l*4 + nb holds at bits 16h + 4g + 2t the row
 *     (0..3, increasing in t) of kept code 2g + t within its group.
 *
 * Errors: as marlin_pack_weights.
 */
marlin_status_t marlin_pack_sparse_weights(const uint8_t *q, const uint16_t *s,
                                           int64_t K, int64_t N, int64_t group,
                                           void *w_packed, void *s_packed,
                                           hipStream_t stream);

/*
 * marlin_unpack_sparse_weights - inverse of marlin_pack_sparse_weights: q
 * receives the dense codes (code 8 at the rows not kept), s the scales.
 * pack followed by unpack is exact for codes with at most two non-8 codes
 * per group of 4 rows.  Errors: as marlin_unpack_weights.
 */
marlin_status_t marlin_unpack_sparse_weights(const void *w_packed, const void *s_packed,
                                             int64_t K, int64_t N, int64_t group,
                                             uint8_t *q, uint16_t *s, hipStream_t stream);

/*
 * marlin_gemm_sparse - C = A * dequant(W) for 2:4 sparse packed weights
 * (Section 4).  Arguments, workspace rules (marlin_workspace_bytes covers
 * both entry points), accumulation, errors and reproducibility: as
 * marlin_gemm, with w_packed in the sparse layout.
 */
marlin_status_t marlin_gemm_sparse(const uint16_t *A, const void *w_packed,
                                   const void *s_packed, uint16_t *C,
                                   void *workspace, size_t workspace_bytes,
                                   int64_t M, int64_t N, int64_t K, int64_t group,
                                   hipStream_t stream);

/* marlin_describe_sparse - as marlin_describe, for marlin_gemm_sparse. */
marlin_status_t marlin_describe_sparse(int64_t M, int64_t N, int64_t K, int64_t group,
                                       char *buf, size_t buf_bytes);

/*
 * ---- Quantiser (Section 2.2, Eq. 1, symmetric; Section 3.5 clipping) ----
 *
 * marlin_quantize - fp16 weights W [K][N] -> codes q and scales s in the
 * format of marlin_pack_weights (w = s * (q - 8)).
 *
 * Each group of `group` consecutive rows of a column (or the whole column,
 * group = -1 or K) is quantised uniformly onto [-a, a] with the fixed zero
 * point 8: s = fp16(2a / 15), q = clamp(rint(v * (1/s)) + 8, 0, 15), the
 * symmetric form of Eq. 1 (Section 2.2) in the format the kernel decodes.
 * The clipping threshold a = r * max|v| is chosen per group among the
 * `n_ratios` ratios r: the one whose reconstruction error
 * sum (v - s (q - 8))^2 (Section 2.2) is smallest, the first one on ties
 * (Section 3.5 names this group-wise clipping search as part of its GPTQ
 * variant; GPTQ's calibration-data updates are not part of this call).
 * A group whose scale rounds to 0 in fp16 gets s = 0 and every code 8.
 * All arithmetic is fp32 in a fixed order (sequential sum over the group's
 * rows, no contracted multiply-adds), so the output is bit-for-bit a
 * function of the input.
 *
 *   W          device, fp16 [K][N] row-major, read only; finite values.
 *   ratios     HOST, n_ratios fp32 values in (0, 1], read during the call
 *              (e.g. {1} for plain round-to-nearest, or 1, 0.95, ..., 0.55).
 *   n_ratios   1..64.
 *   q          device, uint8 [K][N], written (values 0..15).
 *   s          device, fp16 [G][N], written (G = K / group).
 * Shapes and groups as for marlin_pack_weights.  No workspace.
 * Errors: NULL_POINTER, INVALID_SHAPE, UNSUPPORTED_GROUP, MISALIGNED,
 * INVALID_ARGUMENT (n_ratios or a ratio out of range), HIP.
 */
marlin_status_t marlin_quantize(const uint16_t *W, int64_t K, int64_t N, int64_t group,
                                const float *ratios, int n_ratios, uint8_t *q, uint16_t *s,
                                hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MARLIN_MI355X_H */
