/*
 * sbvr.h -- C ABI of the MI355X (gfx950) SBVR GEMV library.
 *
 * SBVR (Summation of BitVector Representation; Bang et al., Sec. 4.1) stores
 * each group of 128 consecutive weights along the inner-product dimension as
 * k bitvectors ("planes") plus k coefficients, so that every decoded weight is
 * a subset sum of its group's coefficients:
 *
 *     w_hat[o][128 g + j] = sum_{i<k} c[o][g][i] * b[o][g][i][j]      (Sec. 4.1)
 *
 * and the GEMV is computed directly on that representation (Sec. 4.4):
 *
 *     y[o] = sum_g sum_i c[o][g][i] * (sum_{j : b[o][g][i][j] = 1} x[128 g + j])
 *
 * Activations x and outputs y are IEEE binary16; accumulation is binary32;
 * y is rounded to binary16 to nearest-even.
 *
 * CANONICAL FORMAT (host-independent, what an encoder writes):
 *   planes  uint32_t [O][G][k][4], G = I / 128.  Bit t (LSB = 0) of word w is
 *           element j = 32 w + t of the group.  Plane i pairs with coefficient
 *           i.  (The paper stores bitvectors "partitioned into 32-bit
 *           integers" in one contiguous tensor, Sec. 4.4.)
 *   coeffs  uint16_t [O][G][k], binary16 bit patterns of c[o][g][i].  The
 *           per-(row, group, plane) coefficient tensor holds the values the
 *           paper's coefficient cache + index (Sec. 4.4) decode to; that
 *           format itself has its own entry points below.
 *
 * DEVICE FORMAT: an opaque, padded repacking of the canonical tensors that
 * the GEMV kernels stream with 128-bit coalesced loads.  It is produced by
 * sbvr_pack and inverted bit-exactly by sbvr_unpack; its size comes from the
 * two size queries.  Its layout is private to the library and may change.
 *
 * CONVENTIONS for every entry point:
 *   - O (out_features) >= 1; I (in_features) >= 128 and a multiple of 128;
 *     1 <= k <= 4 planes; 1 <= B <= 8 activation vectors.
 *   - Pointers named *_dev, x, y, X, Y, planes_canon and coeffs_canon are
 *     device pointers (HIP global memory) owned by the caller.  The library
 *     never allocates, frees or synchronises; work is enqueued on `stream`
 *     (0 = the null stream) and completes asynchronously.  Every call is
 *     safe to capture in a HIP graph.
 *   - Alignment: planes_dev, coeffs_dev, planes_canon, x and X 16 bytes;
 *     coeffs_canon, y and Y 2 bytes.
 *   - On any error nothing is enqueued and no output is written.  No call
 *     aborts, throws or prints.
 *   - Inputs are assumed finite.  Calls on one stream are ordered; calls that
 *     run concurrently on different streams must not share an output buffer.
 */
#ifndef SBVR_H
#define SBVR_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes.  Every entry point returns one of these. */
enum sbvr_status {
    SBVR_OK = 0,
    SBVR_E_INVALID_ARG = -1, /* null pointer, bad shape, B out of range */
    SBVR_E_UNSUPPORTED = -2, /* valid SBVR parameters this build does not run (k > 4) */
    SBVR_E_WORKSPACE = -3,   /* workspace smaller than sbvr_workspace_bytes */
    SBVR_E_ALIGNMENT = -4,   /* a pointer violates the alignment above */
    SBVR_E_HIP = -5          /* the HIP runtime reported a launch error */
};

/* Human-readable name of a status code; never NULL, static storage. */
const char *sbvr_status_string(int status);

/* Library ABI version (major * 100 + minor); 1.01 adds sbvr_decompress,
 * 1.02 sbvr_gemv_a8, 1.03 the coefficient-cache format entry points,
 * 1.04 sbvr_encode and sbvr_decompress_indexed, 1.05 sbvr_gemm_prefill,
 * 1.06 sbvr_gemv_grouped and sbvr_gemv_grouped_a8, 1.07 sbvr_encode_cached. */
int sbvr_version(void);

/*
 * Size queries (pure host functions, no HIP calls).  Bytes the caller must
 * provide for the device planes / device coefficients of an O x I matrix
 * with k planes (the k bitvectors and k coefficients per 128-weight group of
 * Sec. 4.1, stored as in Sec. 4.4, plus the device layout's zero padding of
 * the last row tile and the last 512-element block); 0 if the arguments are
 * invalid.
 */
size_t sbvr_packed_plane_bytes(int O, int I, int k);
size_t sbvr_packed_coeff_bytes(int O, int I, int k);

/*
 * Workspace a GEMV call needs, in bytes (0 means none: pass workspace = NULL
 * and ws_bytes = 0).  The inner-product sum of Sec. 4.4 is split over the
 * wavefronts of one workgroup and reduced there, so the current kernels need
 * no global workspace.
 */
size_t sbvr_workspace_bytes(int O, int I, int k, int B);

/*
 * Repack canonical SBVR tensors into the device format (the storage of
 * Sec. 4.4, laid out for the GEMV kernels).
 *   planes_canon  uint32 [O][G][k][4], coeffs_canon uint16 [O][G][k]: input.
 *   planes_dev    >= sbvr_packed_plane_bytes(O, I, k) bytes: output.
 *   coeffs_dev    >= sbvr_packed_coeff_bytes(O, I, k) bytes: output.
 * Every byte of both outputs is written (padding with zeros).  Inputs and
 * outputs must not overlap.
 */
int sbvr_pack(int O, int I, int k, const uint32_t *planes_canon, const uint16_t *coeffs_canon,
              void *planes_dev, void *coeffs_dev, hipStream_t stream);

/*
 * Inverse of sbvr_pack: recover the canonical tensors (the bitvectors and
 * coefficients of Sec. 4.1 in the storage order of Sec. 4.4), bit for bit,
 * from the device format.  Same shapes and ownership as sbvr_pack with the
 * roles of input and output exchanged.
 */
int sbvr_unpack(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                uint32_t *planes_canon, uint16_t *coeffs_canon, hipStream_t stream);

/*
 * Batch-1 SBVR GEMV (Sec. 4.4 with binary16 activations):
 *     y[o] = fp16_rne( sum_g sum_i c[o][g][i] * sum_j b[o][g][i][j] x[128 g + j] )
 *   planes_dev, coeffs_dev  device-format weights from sbvr_pack.
 *   x  binary16 [I] (input);  y  binary16 [O] (output, every element written).
 *   workspace / ws_bytes    see sbvr_workspace_bytes (may be NULL / 0).
 * x must not overlap y.
 */
int sbvr_gemv(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
              const uint16_t *x, uint16_t *y, void *workspace, size_t ws_bytes,
              hipStream_t stream);

/*
 * Small-batch SBVR GEMM: the GEMV of Sec. 4.4 applied to each of the B
 * activation vectors X[b][0..I) (the paper's kernel handles one token per
 * decode step; a batch of B tokens multiplies the same SBVR weights B times),
 *     Y[b][o] = fp16_rne( sum_g sum_i c[o][g][i] * sum_j b[o][g][i][j] X[b][128 g + j] ),
 * with the weights read from memory once for all B.
 *   X  binary16 [B][I] row-major (input);  Y  binary16 [B][O] row-major
 *   (output, every element written).  1 <= B <= 8.  workspace / ws_bytes as
 *   sbvr_gemv.  X must not overlap Y.
 */
int sbvr_gemm_small_batch(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                          const uint16_t *X, uint16_t *Y, int B, void *workspace,
                          size_t ws_bytes, hipStream_t stream);

/*
 * The W4A8 decode GEMV (Sec. 4.3 and 4.4 with 8-bit SBVR activations): x is
 * converted online, per 128-element group g, to an 8-bit code with Eq. 12's
 * two's-complement coefficients {-128 s_g, s_g, 2 s_g, ..., 64 s_g}:
 *     s_g = max_j abs(x[128 g + j]) / 127,  q_j = rne(x_j / s_g) in [-127, 127]
 * (binary32, correctly rounded division; a zero group has s_g = 0, q = 0),
 * and
 *     y[o] = fp16_rne( sum_g s_g sum_i c[o][g][i] * sum_j b[o][g][i][j] q_j ).
 * Arguments as sbvr_gemv (x binary16 [I], y binary16 [O]).
 */
int sbvr_gemv_a8(int O, int I, int k, const void *planes_dev, const void *coeffs_dev,
                 const uint16_t *x, uint16_t *y, void *workspace, size_t ws_bytes,
                 hipStream_t stream);

/* Most GEMVs one sbvr_gemv_grouped call takes. */
#define SBVR_GEMV_GROUP_MAX 4

/*
 * Grouped batch-1 GEMV: n independent GEMVs of Sec. 4.4 (each exactly the
 * sbvr_gemv of its arguments, bit for bit) enqueued as ONE kernel launch, for
 * the projections of a decode step that run back to back -- e.g. q, k and v,
 * or gate and up, each with its own packed weights -- so that a captured
 * decode step (the paper runs it under a CUDA graph, Sec. 5.2) pays one
 * launch instead of n.
 *   n                 1 <= n <= SBVR_GEMV_GROUP_MAX.
 *   O                 host array [n]: out_features of member i.
 *   I, k              shared by every member.
 *   planes_dev, coeffs_dev, x, y
 *                     host arrays [n] of device pointers, member i's
 *                     device-format weights (sbvr_pack of O[i] x I, k),
 *                     binary16 x[i] [I] (input) and y[i] [O[i]] (output,
 *                     every element written).  Same alignment as sbvr_gemv.
 *   workspace / ws_bytes  as sbvr_gemv (may be NULL / 0).
 * The host arrays are read during the call only.  Members may share an x;
 * no y may overlap another member's y or any x.  Every member is validated
 * as sbvr_gemv would validate it before anything is enqueued; the first
 * failing member's status is returned.
 */
int sbvr_gemv_grouped(int n, const int *O, int I, int k, const void *const *planes_dev,
                      const void *const *coeffs_dev, const uint16_t *const *x, uint16_t *const *y,
                      void *workspace, size_t ws_bytes, hipStream_t stream);

/*
 * The same grouping for the W4A8 decode GEMV: n independent sbvr_gemv_a8
 * calls (Sec. 4.3 and 4.4 with 8-bit SBVR activations, each member bit for
 * bit its own sbvr_gemv_a8) as one kernel launch.  Arguments, ownership and
 * errors as sbvr_gemv_grouped.
 */
int sbvr_gemv_grouped_a8(int n, const int *O, int I, int k, const void *const *planes_dev,
                         const void *const *coeffs_dev, const uint16_t *const *x, uint16_t *const *y,
                         void *workspace, size_t ws_bytes, hipStream_t stream);

/*
 * Prefill GEMM on SBVR weights (the prefill design of Sec. 5.1: the weights
 * are decompressed to binary16 and multiplied on the matrix cores), for a
 * prompt of T tokens, without writing the decompressed matrix to memory:
 *     Y[t][o] = fp16_rne( sum_j X[t][j] * fp16_rne(w_hat[o][j]) ),
 * where fp16_rne(w_hat[o][j]) is the correctly rounded subset sum of
 * Sec. 4.1 (the value sbvr_decompress writes); binary32 accumulation.
 *   planes_dev, coeffs_dev  device-format weights from sbvr_pack.
 *   X  binary16 [T][I] row-major (input, 16-byte aligned);
 *   Y  binary16 [T][O] row-major (output, every element written).
 *   1 <= T <= 2^22 (larger: SBVR_E_UNSUPPORTED).  X must not overlap Y.
 *   The summation order is fixed for given (O, I, k, T), so repeated calls
 *   give identical bits; it follows the launch shape, which depends on T.
 */
int sbvr_gemm_prefill(int O, int I, int k, const void *planes_dev, const void *coeffs_dev, const uint16_t *X,
                      uint16_t *Y, int T, hipStream_t stream);

/*
 * COEFFICIENT-CACHE FORMAT (Sec. 4.4): the coefficients are stored once per
 * distinct coefficient set in a cache, and each (row, group) names the set
 * its k bitvectors use:
 *   planes  uint32_t [O][G][k][4] as in the canonical format;
 *   index   uint16_t [O][G]: coefficient-set index of (row o, group g);
 *   table   uint16_t [n_sets][k]: binary16 coefficient sets, 1 <= n_sets <= 65536;
 *     c[o][g][i] = table[index[o][g]][i].
 * Per weight this stores 2 bytes per group instead of 2k (k = 4: 4.125
 * instead of 4.5 bits per weight) plus the table.  An index >= n_sets is a
 * caller error; the GEMV then reads zero coefficients for that group (the
 * table is read through a bounds-checked path), nothing faults.
 */

/* Device bytes of the index blocks of an O x I matrix with k planes, and of
 * a table of n_sets coefficient sets (8 bytes per set); 0 if invalid. */
size_t sbvr_packed_index_bytes(int O, int I, int k);
size_t sbvr_packed_table_bytes(int n_sets, int k);

/*
 * Repack the coefficient-cache format into its device format.
 *   planes_canon uint32 [O][G][k][4], index_canon uint16 [O][G],
 *   table_canon uint16 [n_sets][k]: inputs (device memory; planes_canon
 *   16-byte aligned, the others 2).
 *   planes_dev (sbvr_packed_plane_bytes), index_dev
 *   (sbvr_packed_index_bytes), table_dev (sbvr_packed_table_bytes): outputs,
 *   16-byte aligned, every byte written.  Inputs and outputs must not overlap.
 */
int sbvr_pack_indexed(int O, int I, int k, int n_sets, const uint32_t *planes_canon,
                      const uint16_t *index_canon, const uint16_t *table_canon, void *planes_dev,
                      void *index_dev, void *table_dev, hipStream_t stream);

/* Inverse of sbvr_pack_indexed, bit for bit (roles of inputs and outputs
 * exchanged). */
int sbvr_unpack_indexed(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                        const void *table_dev, uint32_t *planes_canon, uint16_t *index_canon,
                        uint16_t *table_canon, hipStream_t stream);

/*
 * Batch-1 GEMV on the coefficient-cache format (Sec. 4.4):
 *     y[o] = fp16_rne( sum_g sum_i table[index[o][g]][i] * sum_j b[o][g][i][j] x[128 g + j] )
 * i.e. sbvr_gemv with the gathered coefficients.  planes_dev, index_dev,
 * table_dev from sbvr_pack_indexed; x, y, workspace as sbvr_gemv.
 */
int sbvr_gemv_indexed(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                      const void *table_dev, const uint16_t *x, uint16_t *y, void *workspace,
                      size_t ws_bytes, hipStream_t stream);

/*
 * The same with SBVR-8 activations (the conversion of sbvr_gemv_a8): the
 * paper's decode configuration, W4A8 with a coefficient cache (Sec. 4.3-4.4).
 */
int sbvr_gemv_indexed_a8(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                         const void *table_dev, const uint16_t *x, uint16_t *y, void *workspace,
                         size_t ws_bytes, hipStream_t stream);

/*
 * Decompression for the prefill path: the decoded matrix as binary16,
 *     W[o][128 g + j] = fp16_rne( sum_i c[o][g][i] * b[o][g][i][j] )
 * (the subset-sum decoding of Sec. 4.1, computed exactly and rounded once),
 * for a dense matrix-core GEMM over many tokens.
 *   planes_dev, coeffs_dev  device-format weights from sbvr_pack.
 *   W  binary16 [O][I] row-major (output, every element written), 16-byte
 *      aligned; must not overlap the inputs.
 */
int sbvr_decompress(int O, int I, int k, const void *planes_dev, const void *coeffs_dev, uint16_t *W,
                    hipStream_t stream);

/*
 * Prefill decompression of the coefficient-cache format: as sbvr_decompress
 * with c[o][g][i] = table[index[o][g]][i] (zero for an index >= n_sets).
 * planes_dev, index_dev, table_dev from sbvr_pack_indexed; W as for
 * sbvr_decompress.
 */
int sbvr_decompress_indexed(int O, int I, int k, int n_sets, const void *planes_dev, const void *index_dev,
                            const void *table_dev, uint16_t *W, hipStream_t stream);

#define SBVR_ENCODE_MAX_ENTRIES 65536

/*
 * SBVR encoding on the GPU (Algorithm 1 and the bitvector assignment of
 * Sec. 4.2): every 128-weight group of W takes, from the (r, s, b) grid of
 * Eqs. 4-11 with |R1| = n_ratio1, |R2| = n_ratio2, N_scale = n_scale and
 * N_bias = n_bias entries, the binary16 coefficient set with the smallest
 * mean squared error of nearest-subset-sum reconstruction (first such entry
 * in (r, s, b) order), and each weight the bit pattern of its nearest subset
 * sum (lowest pattern index on ties).  normalise = 1 divides the geometric
 * series of Eq. 4 by sum_i abs(r)^i (the span-normalised reading), 0 takes
 * Eq. 4 literally.  Groups with no admissible entry (s <= 0 or a non-finite
 * coefficient everywhere) get (fp16(mean), 0, ...).  All arithmetic is
 * binary64 in a fixed order, so the output is deterministic and reproducible
 * bit for bit by a CPU implementation of the same definition.
 *   W             float32 [O][I] row-major, device, 4-byte aligned; finite.
 *   planes_canon  uint32 [O][G][k][4] canonical planes (output, 16-byte aligned).
 *   coeffs_canon  uint16 [O][G][k] binary16 coefficients (output).
 *   mse           binary64 [O][G] (output, 8-byte aligned) or NULL.
 * At most SBVR_ENCODE_MAX_ENTRIES grid entries ((n_ratio1 + n_ratio2) *
 * n_scale * n_bias); more is SBVR_E_UNSUPPORTED.
 */
int sbvr_encode(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                int normalise, uint32_t *planes_canon, uint16_t *coeffs_canon, double *mse,
                hipStream_t stream);

#define SBVR_ENCODE_CACHE_MAX 64

/*
 * The encoder with the cache of Sec. 4.2 (last paragraph and its footnote):
 * before the full search, a group tries the coefficient sets that the search
 * chose for earlier groups, and keeps one if its error is below the moving
 * average of the quantization error; groups that hit share their set with an
 * earlier group, which also shrinks the coefficient cache of the indexed
 * format (sbvr_pack_indexed).  Each row of W is encoded on its own, its
 * groups in index order:
 *   - the cache holds the coefficient sets the full search chose for the
 *     row's last cache_slots searched groups (the oldest is replaced first;
 *     the (fp16(mean), 0, ...) fallback is not cached);
 *   - every held set is scored on the group with the search's MSE; the
 *     smallest (the oldest set among equal ones) is taken, with each weight's
 *     nearest-subset-sum pattern, if it is strictly below the mean MSE of
 *     the row's earlier groups (binary64 sum in group order over their count);
 *   - otherwise the group runs the search of sbvr_encode, and its set enters
 *     the cache.
 * The first group of a row always searches; cache_slots = 0 gives exactly
 * sbvr_encode's output.  Arguments as sbvr_encode, plus
 *   cache_slots  0 .. SBVR_ENCODE_CACHE_MAX (else SBVR_E_INVALID_ARG).
 *   hits         uint8 [O][G] (output): 1 where the group took a cached set,
 *                0 where it searched; or NULL.
 * Rows are independent (one wavefront each), a row's groups sequential.
 */
int sbvr_encode_cached(int O, int I, int k, const float *W, int n_ratio1, int n_ratio2, int n_scale, int n_bias,
                       int normalise, int cache_slots, uint32_t *planes_canon, uint16_t *coeffs_canon,
                       double *mse, uint8_t *hits, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SBVR_H */
